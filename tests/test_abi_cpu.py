"""Host-side tests of the C ABI (no GPU needed): the library loads and exports
every function include/slorr.h declares, the library's schedule generator
agrees with the oracle's independent one, plans report the right facts, and
every argument error is reported before anything touches a device.
"""
import ctypes
import math
import os
import re

import numpy as np
import pytest

from oracle.pe_schedule import pe_schedule
from workloads import CONFIGS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    import paper_2607_08754_amd._lib as lib_mod
    return lib_mod


def _declared_functions():
    text = open(os.path.join(ROOT, "include", "slorr.h")).read()
    return sorted(set(re.findall(r"SLORR_API\s+[\w\s\*]*?\b(slorr_\w+)\s*\(", text)))


def test_exports_match_header(L):
    declared = _declared_functions()
    assert len(declared) >= 10
    lib = L.lib()
    for name in declared:
        assert hasattr(lib, name), name
    assert sorted(L.EXPORTED) == declared
    out = os.popen(f"nm -D --defined-only {L.LIB_PATH}").read()
    exported = sorted(set(re.findall(r"\bT (slorr_\w+)", out)))
    assert exported == declared                      # nothing else is exported


def test_schedule_matches_oracle(L):
    """Two independent Remez implementations (C++ library, NumPy oracle)."""
    from paper_2607_08754_amd import pe_coefficients
    for ell in (1e-3, 0.05, 0.3):
        for d in (3, 5):
            lib_tab = pe_coefficients(8, ell, d)
            ora_tab = pe_schedule(8, ell, d)
            # rows solved on narrow intervals (half-width ~1e-3) are limited by
            # the conditioning of the Remez system, not by the method
            assert np.allclose(lib_tab, ora_tab, rtol=1e-10, atol=1e-10), (ell, d)
    # the paper's setting, T = 6: wide intervals, agreement to rounding
    assert np.allclose(pe_coefficients(6), pe_schedule(6), rtol=1e-13, atol=0)


def _plan(L, shapes, dtype=0, kind=0, opts=None):
    lib = L.lib()
    h = ctypes.c_void_p()
    ws = ctypes.c_size_t()
    arr = (L.Shape * max(1, len(shapes)))(*[L.Shape(r, c) for r, c in shapes])
    st = lib.slorr_plan(ctypes.byref(h), len(shapes), arr, dtype, kind,
                        ctypes.byref(opts) if opts is not None else None, ctypes.byref(ws))
    return st, h, ws.value, arr


def _pad(x):
    return (x + 127) // 128 * 128


def _tri(P, t):
    nt = P // t
    return nt * (nt + 1) / 2 * float(t) * t


def _expected_mfma(shapes, T):
    """MFMA work of the schedule. Per step: A = X X^T on upper-triangle tiles
    (256 x 256 when every matrix is 256-aligned and the launch has one such
    tile per CU; else 128 x 128, split into k parts when there are fewer than
    two tiles per CU: the parts cover each k once, so the work is the same),
    the poly on upper-triangle tiles (256 x 256 from two per CU), B X on all
    tiles (its work does not depend on the tile edge)."""
    mats = [(_pad(min(s)), _pad(max(s))) for s in shapes if min(s) > 0]

    def cfg(ps, min_big):
        big = sum((P // 256) * (P // 256 + 1) // 2 for P in ps)
        return 256 if ps and all(P % 256 == 0 for P in ps) and big >= min_big else 128

    ps = [P for P, _ in mats]
    tg, tp = cfg(ps, 256), cfg(ps, 512)
    return T * sum(2 * _tri(P, tg) * Q + 2 * _tri(P, tp) * P + 2.0 * P * P * Q for P, Q in mats)


def _split_k(shapes, dtype="bf16"):
    """Whether the Gram launch is split into k parts: 128-tiles, fewer than
    512 of them, and a longest tile of at least 32 k-slabs of 64 values of k
    (the fp16 iterate of bf16 sets) or 8 k-slabs of 32 values (fp32 sets)."""
    mats = [(_pad(min(s)), _pad(max(s))) for s in shapes if min(s) > 0]
    big = sum((P // 256) * (P // 256 + 1) // 2 for P, _ in mats)
    if mats and all(P % 256 == 0 for P, _ in mats) and big >= 256:
        return False
    slab, need = (64, 32) if dtype == "bf16" else (32, 8)
    if not mats or max(Q for _, Q in mats) // slab < need:
        return False
    n128 = sum((P // 128) * (P // 128 + 1) // 2 for P, _ in mats)
    return 0 < n128 < 512


@pytest.mark.parametrize("name", list(CONFIGS))
def test_plan_facts(L, name):
    cfg = CONFIGS[name]
    lib = L.lib()
    opts = L.Options()
    lib.slorr_default_options(ctypes.byref(opts))
    opts.iters = cfg.iters
    st, h, ws, _ = _plan(L, cfg.shapes, L.BF16 if cfg.dtype == "bf16" else L.F32, L.HOYER, opts)
    assert st == L.OK, lib.slorr_last_error()
    info = L.PlanInfo()
    assert lib.slorr_plan_get_info(h, ctypes.byref(info)) == L.OK
    assert info.n == cfg.n and info.iters == cfg.iters
    assert info.paper_flops == pytest.approx(cfg.flops(), rel=1e-12)
    assert info.mfma_flops == pytest.approx(_expected_mfma(cfg.shapes, cfg.iters), rel=1e-12)
    assert info.mfma_flops <= info.paper_flops * (1.0 if name in ("vit_b16", "vit_l16", "llm560") else 4.0)
    assert info.groups == len({(min(s), max(s)) for s in cfg.shapes})
    # sumsq, norm, prep; per step the Gram (+ its reduce when split), the poly
    # and the update; finalize, grad (its first block writes the set total)
    per_step = 4 if _split_k(cfg.shapes, cfg.dtype) else 3
    assert info.launches == 3 + per_step * cfg.iters + 2
    assert info.workspace_bytes == ws > 0
    esz = 2 if cfg.dtype == "bf16" else 4
    assert info.weight_bytes == sum(r * c * esz for r, c in cfg.shapes)
    assert lib.slorr_plan_destroy(h) == L.OK


def test_plan_launch_work(L):
    """slorr_plan_get_launches: one kind per launch, algorithmic flops of the
    products each performs; over a call T (2 P^2 Q + 2 P^3 + 2 P^2 Q), the
    paper's count (Sec. 3 "Computational cost")."""
    lib = L.lib()
    opts = L.Options()
    for name in ("tiny", "resnet18", "vit_b16", "llm560"):
        cfg = CONFIGS[name]
        lib.slorr_default_options(ctypes.byref(opts))
        st, h, _, _ = _plan(L, cfg.shapes, L.BF16 if cfg.dtype == "bf16" else L.F32, L.HOYER, opts)
        assert st == L.OK
        info = L.PlanInfo()
        lib.slorr_plan_get_info(h, ctypes.byref(info))
        nl = info.launches
        ops = (ctypes.c_int32 * nl)()
        fl = (ctypes.c_double * nl)()
        te = (ctypes.c_int32 * nl)()
        assert lib.slorr_plan_get_launches(h, ops, fl, te) == L.OK
        names = [L.OPS[o] for o in ops]
        gemm = ("gram", "poly", "update", "last")
        assert all((e in (128, 256)) if o in gemm else e == 0 for o, e in zip(names, te))
        assert names[:3] == ["sumsq", "norm", "prep"] and names[-2:] == ["finalize", "grad"]
        assert "setsum" not in names                       # written by the gradient launch
        T = info.iters                                     # the default options: T = 6
        assert names.count("last") == 1 and names.count("update") == T - 1 and names.count("poly") == T
        want = sum(T * (4.0 * min(s) ** 2 * max(s) + 2.0 * min(s) ** 3) for s in cfg.shapes)
        assert sum(fl) == pytest.approx(want, rel=1e-12)
        assert all(f == 0.0 for f, o in zip(fl, names) if o not in gemm)
        assert lib.slorr_plan_get_launches(h, None, None, None) == L.OK
        lib.slorr_plan_destroy(h)
    assert lib.slorr_plan_get_launches(None, None, None, None) == L.ERR_INVALID_ARGUMENT


def test_empty_plans(L):
    st, h, ws, _ = _plan(L, [])
    assert st == L.OK and ws > 0
    L.lib().slorr_plan_destroy(h)
    st, h, ws, _ = _plan(L, [(0, 7), (5, 0)])
    assert st == L.OK
    info = L.PlanInfo()
    L.lib().slorr_plan_get_info(h, ctypes.byref(info))
    assert info.launches == 3 and info.gemm_tiles == 0       # norm + finalize + set sum
    L.lib().slorr_plan_destroy(h)


def test_plan_errors(L):
    lib = L.lib()
    h = ctypes.c_void_p(1234)
    ws = ctypes.c_size_t()
    one = (L.Shape * 1)(L.Shape(4, 8))
    # null out-pointers / shapes, negative n
    assert lib.slorr_plan(None, 1, one, 0, 0, None, ctypes.byref(ws)) == L.ERR_INVALID_ARGUMENT
    assert lib.slorr_plan(ctypes.byref(h), 1, one, 0, 0, None, None) == L.ERR_INVALID_ARGUMENT
    assert h.value is None                                    # set to NULL on error
    assert lib.slorr_plan(ctypes.byref(h), 1, None, 0, 0, None, ctypes.byref(ws)) == L.ERR_INVALID_ARGUMENT
    assert lib.slorr_plan(ctypes.byref(h), -1, one, 0, 0, None, ctypes.byref(ws)) == L.ERR_INVALID_ARGUMENT
    assert b"n must be" in lib.slorr_last_error()
    # bad shapes
    for r, c, want in [(-1, 4, L.ERR_INVALID_ARGUMENT), (16385, 16385, L.ERR_UNSUPPORTED),
                       (4, (1 << 20) + 1, L.ERR_UNSUPPORTED), (16384, 1 << 20, L.ERR_UNSUPPORTED)]:
        st, _, _, _ = _plan(L, [(r, c)])
        assert st == want, (r, c, st)
    # the padded canonical matrix must stay under 2 GiB in the iterate type
    # (fp32 sets: 4 bytes, bf16 sets: 2 bytes per element)
    for r, c, dt, want in [(16384, 32768, 0, L.ERR_UNSUPPORTED), (16300, 32700, 0, L.ERR_UNSUPPORTED),
                           (32640, 16384, 0, L.OK), (16384, 65536, 1, L.ERR_UNSUPPORTED), (16384, 65408, 1, L.OK)]:
        st, h, _, _ = _plan(L, [(r, c)], dtype=dt)
        assert st == want, (r, c, dt, st)
        if st == L.OK:
            assert lib.slorr_plan_destroy(h) == L.OK
        else:
            assert b"2 GiB" in lib.slorr_last_error()
    # dtype / kind
    assert _plan(L, [(4, 8)], dtype=7)[0] == L.ERR_UNSUPPORTED
    assert _plan(L, [(4, 8)], kind=9)[0] == L.ERR_UNSUPPORTED
    # options
    def with_opts(**kw):
        o = L.Options()
        lib.slorr_default_options(ctypes.byref(o))
        for k, v in kw.items():
            setattr(o, k, v)
        return _plan(L, [(4, 8)], opts=o)[0]
    assert with_opts(iters=-2) == L.ERR_INVALID_ARGUMENT
    assert with_opts(iters=5000) == L.ERR_INVALID_ARGUMENT
    assert with_opts(degree=7) == L.ERR_UNSUPPORTED
    assert with_opts(ell=1.5) == L.ERR_INVALID_ARGUMENT
    assert with_opts(ell=-0.1) == L.ERR_INVALID_ARGUMENT
    assert with_opts(eps=-1.0) == L.ERR_INVALID_ARGUMENT
    assert with_opts(eps=float("inf")) == L.ERR_INVALID_ARGUMENT
    assert with_opts(flags=0x100) == L.ERR_INVALID_ARGUMENT
    assert with_opts(flags=0x20) == L.ERR_INVALID_ARGUMENT      # no such flag
    bad = (ctypes.c_double * 18)(*([1.0] * 17 + [float("nan")]))
    assert with_opts(coeffs=ctypes.cast(bad, ctypes.POINTER(ctypes.c_double))) == L.ERR_INVALID_ARGUMENT
    assert with_opts() == L.OK


def test_pe_coefficients_errors(L):
    lib = L.lib()
    out = (ctypes.c_double * 30)()
    assert lib.slorr_pe_coefficients(1e-3, 5, 6, None) == L.ERR_INVALID_ARGUMENT
    assert lib.slorr_pe_coefficients(1e-3, 4, 6, out) == L.ERR_UNSUPPORTED
    assert lib.slorr_pe_coefficients(0.0, 5, 6, out) == L.ERR_INVALID_ARGUMENT
    assert lib.slorr_pe_coefficients(1e-3, 5, 0, out) == L.ERR_INVALID_ARGUMENT
    assert lib.slorr_pe_coefficients(1e-3, 5, 10, out) == L.OK


def test_call_errors_before_any_device_use(L):
    """Argument checks of slorr_reg_fwd_bwd run before the workspace check and
    before any HIP call, so they are testable on a machine without a GPU."""
    lib = L.lib()
    st, h, ws, shapes = _plan(L, [(4, 8), (8, 4)])
    assert st == L.OK
    vals = ctypes.c_void_p(0x10000)
    w = (ctypes.c_void_p * 2)(0x20000, 0x30000)
    g = (ctypes.c_void_p * 2)(0x40000, 0x50000)
    call = lib.slorr_reg_fwd_bwd
    assert call(h, 3, w, shapes, 0, 6, vals, g, 1.0, None) == L.ERR_PLAN_MISMATCH
    assert call(h, 2, w, shapes, 1, 6, vals, g, 1.0, None) == L.ERR_PLAN_MISMATCH
    assert call(h, 2, w, shapes, 0, 5, vals, g, 1.0, None) == L.ERR_PLAN_MISMATCH
    other = (L.Shape * 2)(L.Shape(4, 8), L.Shape(4, 8))
    assert call(h, 2, w, other, 0, 6, vals, g, 1.0, None) == L.ERR_PLAN_MISMATCH
    assert call(h, 2, w, shapes, 0, 6, None, g, 1.0, None) == L.ERR_INVALID_ARGUMENT
    assert call(h, 2, w, shapes, 0, 6, ctypes.c_void_p(0x10001), g, 1.0, None) == L.ERR_INVALID_ARGUMENT
    assert call(h, 2, None, shapes, 0, 6, vals, g, 1.0, None) == L.ERR_INVALID_ARGUMENT
    assert call(h, 2, w, shapes, 0, 6, vals, None, 1.0, None) == L.ERR_INVALID_ARGUMENT
    misaligned = (ctypes.c_void_p * 2)(0x20008, 0x30000)
    assert call(h, 2, misaligned, shapes, 0, 6, vals, g, 1.0, None) == L.ERR_INVALID_ARGUMENT
    nullw = (ctypes.c_void_p * 2)(0x20000, None)
    assert call(h, 2, nullw, shapes, 0, 6, vals, g, 1.0, None) == L.ERR_INVALID_ARGUMENT
    # gradient 0 (4x8 fp32 = 128 B at 0x40000) overlaps gradient 1
    overlap = (ctypes.c_void_p * 2)(0x40000, 0x40040)
    assert call(h, 2, w, shapes, 0, 6, vals, overlap, 1.0, None) == L.ERR_INVALID_ARGUMENT
    alias = (ctypes.c_void_p * 2)(0x20000, 0x50000)              # grad 0 == weight 0
    assert call(h, 2, w, shapes, 0, 6, vals, alias, 1.0, None) == L.ERR_INVALID_ARGUMENT
    # weights may overlap each other (read only); then: no workspace attached
    shared_w = (ctypes.c_void_p * 2)(0x20000, 0x20000)
    assert call(h, 2, shared_w, shapes, 0, 6, vals, g, 1.0, None) == L.ERR_WORKSPACE
    assert call(h, 2, w, shapes, 0, 6, vals, g, 1.0, None) == L.ERR_WORKSPACE
    assert b"workspace" in lib.slorr_last_error()
    ms = (ctypes.c_float * 32)()
    assert lib.slorr_reg_fwd_bwd_profiled(h, 2, w, shapes, 0, 6, vals, g, 1.0, None, None, None) == L.ERR_INVALID_ARGUMENT
    assert lib.slorr_reg_fwd_bwd_profiled(h, 2, w, shapes, 0, 6, vals, g, 1.0, None, ms, None) == L.ERR_WORKSPACE
    # workspace checks that precede any device call
    assert lib.slorr_plan_set_workspace(h, None, ws) == L.ERR_WORKSPACE
    assert lib.slorr_plan_set_workspace(h, ctypes.c_void_p(0x1000 + 16), ws) == L.ERR_WORKSPACE
    assert lib.slorr_plan_set_workspace(h, ctypes.c_void_p(0x1000), ws - 1) == L.ERR_WORKSPACE
    assert lib.slorr_plan_destroy(h) == L.OK
    assert lib.slorr_plan_destroy(None) == L.OK


def test_values_only_accepts_null_grads(L):
    lib = L.lib()
    o = L.Options()
    lib.slorr_default_options(ctypes.byref(o))
    o.flags = L.VALUES_ONLY
    st, h, _, shapes = _plan(L, [(4, 8)], opts=o)
    assert st == L.OK
    w = (ctypes.c_void_p * 1)(0x20000)
    assert lib.slorr_reg_fwd_bwd(h, 1, w, shapes, 0, 6, ctypes.c_void_p(0x10000), None, 1.0, None) == L.ERR_WORKSPACE
    lib.slorr_plan_destroy(h)


def test_status_strings(L):
    lib = L.lib()
    for code in range(7):
        assert lib.slorr_status_string(code).startswith(b"SLORR_")
    assert lib.slorr_status_string(99) == b"SLORR_UNKNOWN_STATUS"


def test_binding_validates_in_python(L):
    """The Python wrapper rejects mismatched tensors before calling the ABI."""
    from paper_2607_08754_amd import Plan
    p = Plan([(4, 8)], dtype="f32", create_workspace=False)
    with pytest.raises(RuntimeError):
        p([np.zeros((4, 8))], None)
    assert p.info()["n"] == 1
    p.close()


def test_deferred_gradient_and_apply_checks_before_device_use(L):
    lib = L.lib()

    def opts(**kw):
        o = L.Options()
        lib.slorr_default_options(ctypes.byref(o))
        for k, v in kw.items():
            setattr(o, k, v)
        return o
    assert opts().grad_dtype == L.F32
    assert _plan(L, [(4, 8)], opts=opts(flags=L.VALUES_ONLY | L.DEFER_GRAD))[0] == L.ERR_INVALID_ARGUMENT
    assert _plan(L, [(4, 8)], opts=opts(grad_dtype=5))[0] == L.ERR_UNSUPPORTED
    # the deferred plan drops the gradient launch from its schedule
    st, hn, _, _ = _plan(L, [(4, 8), (8, 4)])
    st2, hd, _, shapes = _plan(L, [(4, 8), (8, 4)], opts=opts(flags=L.DEFER_GRAD, grad_dtype=L.BF16))
    assert st == st2 == L.OK
    ni, di = L.PlanInfo(), L.PlanInfo()
    lib.slorr_plan_get_info(hn, ctypes.byref(ni))
    lib.slorr_plan_get_info(hd, ctypes.byref(di))
    # (and writes the set total with a launch of its own instead)
    assert di.launches == ni.launches
    w = (ctypes.c_void_p * 2)(0x20000, 0x30000)
    vals = ctypes.c_void_p(0x10000)
    # forward of a deferred plan needs no gradient buffers
    assert lib.slorr_reg_fwd_bwd(hd, 2, w, shapes, 0, 6, vals, None, 1.0, None) == L.ERR_WORKSPACE
    # bf16 gradients: 4x8 bf16 = 64 B, so these two buffers do not overlap
    g = (ctypes.c_void_p * 2)(0x40000, 0x40040)
    rg = lib.slorr_reg_grad
    assert rg(None, 2, w, shapes, 0, 6, g, None, 1.0, None) == L.ERR_INVALID_ARGUMENT
    assert rg(hd, 3, w, shapes, 0, 6, g, None, 1.0, None) == L.ERR_PLAN_MISMATCH
    assert rg(hd, 2, w, shapes, 0, 6, g, None, 1.0, None) == L.ERR_INVALID_ARGUMENT
    assert b"no forward state" in lib.slorr_last_error()
    ap = lib.slorr_decoupled_apply
    assert ap(None, 2, w, shapes, g, None, 1.0, None) == L.ERR_INVALID_ARGUMENT
    assert ap(hd, 1, w, shapes, g, None, 1.0, None) == L.ERR_PLAN_MISMATCH
    assert ap(hd, 2, w, shapes, None, None, 1.0, None) == L.ERR_INVALID_ARGUMENT
    assert ap(hd, 2, w, shapes, g, ctypes.c_void_p(0x70002), 1.0, None) == L.ERR_INVALID_ARGUMENT
    alias = (ctypes.c_void_p * 2)(0x20000, 0x50000)
    assert ap(hd, 2, w, shapes, alias, None, 1.0, None) == L.ERR_INVALID_ARGUMENT
    assert ap(hd, 2, w, shapes, g, None, 1.0, None) == L.ERR_WORKSPACE
    # the same buffers overlap once the gradients are fp32 (128 B each)
    assert ap(hn, 2, w, shapes, g, None, 1.0, None) == L.ERR_INVALID_ARGUMENT
    # a values-only plan has no gradient to defer
    st3, hv, _, _ = _plan(L, [(4, 8), (8, 4)], opts=opts(flags=L.VALUES_ONLY))
    assert rg(hv, 2, w, shapes, 0, 6, g, None, 1.0, None) == L.ERR_INVALID_ARGUMENT
    assert b"values only" in lib.slorr_last_error()
    for h in (hn, hd, hv):
        lib.slorr_plan_destroy(h)


def test_split_k_gram_plan(L):
    """A set with few but long Gram tiles gets split-K Gram parts plus a
    reduce launch in every step; the parts cover every k exactly once (same
    executed MFMA work as one pass per tile). Sets with enough tiles, or with
    short ones, are not split."""
    def facts(shapes):
        st, h, _, _ = _plan(L, shapes, L.BF16, L.HOYER)
        assert st == L.OK
        info = L.PlanInfo()
        L.lib().slorr_plan_get_info(h, ctypes.byref(info))
        L.lib().slorr_plan_destroy(h)
        return info
    T = 6
    for shapes in ([(384, 2048), (2048, 384), (256, 2304)], [(256, 4096), (4096, 256), (384, 2944)]):
        assert _split_k(shapes)
        info = facts(shapes)
        assert info.launches == 3 + 4 * T + 2                # gram parts, reduce, poly, update
        assert info.mfma_flops == pytest.approx(_expected_mfma(shapes, T), rel=1e-12)
    big = facts(CONFIGS["vit_b16"].shapes)
    assert not _split_k(CONFIGS["vit_b16"].shapes)
    assert big.launches == 3 + 3 * T + 2
    short = [(384, 640), (640, 384), (256, 384)]         # few tiles, but short: one pass
    assert not _split_k(short)
    assert facts(short).launches == 3 + 3 * T + 2


def test_null_plan_checks_before_device_use(L):
    """slorr_reg_fwd_bwd with plan == NULL (the internal plan cache) rejects
    bad arguments before it selects a device or builds a plan; and the cache
    configuration and release entry points need no device."""
    lib = L.lib()
    one = (L.Shape * 1)(L.Shape(4, 8))
    w = (ctypes.c_void_p * 1)(0x20000)
    g = (ctypes.c_void_p * 1)(0x40000)
    vals = ctypes.c_void_p(0x10000)
    call = lib.slorr_reg_fwd_bwd
    lib.slorr_cache_config(L.F32, None)
    assert call(None, -1, w, one, 0, 6, vals, g, 1.0, None) == L.ERR_INVALID_ARGUMENT
    assert call(None, 1, w, None, 0, 6, vals, g, 1.0, None) == L.ERR_INVALID_ARGUMENT
    assert call(None, 1, None, one, 0, 6, vals, g, 1.0, None) == L.ERR_INVALID_ARGUMENT
    assert call(None, 1, w, one, 0, 0, vals, g, 1.0, None) == L.ERR_INVALID_ARGUMENT
    assert call(None, 1, w, one, 0, 6, None, g, 1.0, None) == L.ERR_INVALID_ARGUMENT
    assert call(None, 1, w, one, 0, 6, ctypes.c_void_p(0x10002), g, 1.0, None) == L.ERR_INVALID_ARGUMENT
    assert call(None, 1, w, one, 0, 6, vals, None, 1.0, None) == L.ERR_INVALID_ARGUMENT
    assert b"out_grads" in lib.slorr_last_error()
    o = L.Options()
    lib.slorr_default_options(ctypes.byref(o))
    o.flags = L.VALUES_ONLY
    tab = (ctypes.c_double * 9)(*([1.875, -1.25, 0.375] * 3))
    o.iters = 3
    o.coeffs = ctypes.cast(tab, ctypes.POINTER(ctypes.c_double))
    lib.slorr_cache_config(L.BF16, ctypes.byref(o))          # copies the table
    del tab
    assert call(None, 1, w, one, 0, 6, None, None, 1.0, None) == L.ERR_INVALID_ARGUMENT
    lib.slorr_cache_config(L.F32, None)
    assert lib.slorr_cache_clear() == L.OK                   # empty cache: no device call


def test_noalloc_checks_before_device_use(L):
    """slorr_reg_fwd_bwd_noalloc: argument errors, a plan larger than the static
    scratch and a deferred-gradient plan are refused before any device call."""
    lib = L.lib()
    call = lib.slorr_reg_fwd_bwd_noalloc
    st, h, ws, shapes = _plan(L, [(4, 8), (8, 4)])
    assert st == L.OK
    vals = ctypes.c_void_p(0x10000)
    w = (ctypes.c_void_p * 2)(0x20000, 0x30000)
    g = (ctypes.c_void_p * 2)(0x40000, 0x50000)
    assert call(None, 2, w, shapes, 0, 6, vals, g, 1.0, None) == L.ERR_INVALID_ARGUMENT
    assert call(h, 3, w, shapes, 0, 6, vals, g, 1.0, None) == L.ERR_PLAN_MISMATCH
    assert call(h, 2, w, shapes, 1, 6, vals, g, 1.0, None) == L.ERR_PLAN_MISMATCH
    assert call(h, 2, w, shapes, 0, 6, None, g, 1.0, None) == L.ERR_INVALID_ARGUMENT
    assert call(h, 2, w, shapes, 0, 6, vals, None, 1.0, None) == L.ERR_INVALID_ARGUMENT
    alias = (ctypes.c_void_p * 2)(0x20000, 0x50000)
    assert call(h, 2, w, shapes, 0, 6, vals, alias, 1.0, None) == L.ERR_INVALID_ARGUMENT
    lib.slorr_plan_destroy(h)
    o = L.Options()
    lib.slorr_default_options(ctypes.byref(o))
    o.flags = L.DEFER_GRAD
    st, h, _, shapes = _plan(L, [(4, 8), (8, 4)], opts=o)
    assert call(h, 2, w, shapes, 0, 6, vals, g, 1.0, None) == L.ERR_INVALID_ARGUMENT
    assert b"DEFER_GRAD" in lib.slorr_last_error()
    lib.slorr_plan_destroy(h)
    big = [(1024, 8192)] * 4                       # > 64 MiB of workspace
    st, h, ws, shapes = _plan(L, big, L.BF16)
    assert st == L.OK and ws > (64 << 20)
    w4 = (ctypes.c_void_p * 4)(*[0x100000000 * (i + 1) for i in range(4)])
    g4 = (ctypes.c_void_p * 4)(*[0x800000000 + 0x100000000 * i for i in range(4)])
    assert call(h, 4, w4, shapes, 0, 6, vals, g4, 1.0, None) == L.ERR_WORKSPACE
    assert b"static scratch" in lib.slorr_last_error()
    lib.slorr_plan_destroy(h)
