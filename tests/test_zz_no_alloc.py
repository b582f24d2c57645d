"""The entry point that allocates nothing (slorr_reg_fwd_bwd_noalloc) against
the regular one (slorr_reg_fwd_bwd) through the C ABI: two calls in a row on
plans without a workspace, the second with a smaller set, each compared with
the regular entry point's result on the same inputs (same kernels and
rounding: bitwise)."""
import ctypes

import numpy as np
import pytest

from parity_util import to_device
from workloads import gaussian

pytestmark = pytest.mark.gpu


def _run(dtype, shapes, seed, noalloc, L):
    import torch
    from paper_2607_08754_amd import Plan
    lib = L.lib()
    arrs = [gaussian(s, seed=seed, std=0.05, dtype=dtype, index=i) for i, s in enumerate(shapes)]
    W = to_device(arrs, dtype, "cuda:0")
    G = [torch.full(s, float("nan"), dtype=torch.float32, device="cuda:0") for s in shapes]
    vals = torch.full((len(shapes) + 1,), float("nan"), dtype=torch.float32, device="cuda:0")
    plan = Plan(shapes, dtype=dtype, kind="hoyer", iters=6, eps=1e-4, device="cuda:0",
                create_workspace=not noalloc)
    c_shapes = (L.Shape * len(shapes))(*[L.Shape(r, c) for r, c in shapes])
    wp = (ctypes.c_void_p * len(shapes))(*[w.data_ptr() for w in W])
    gp = (ctypes.c_void_p * len(shapes))(*[g.data_ptr() for g in G])
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    fn = lib.slorr_reg_fwd_bwd_noalloc if noalloc else lib.slorr_reg_fwd_bwd
    st = fn(plan._handle, len(shapes), wp, c_shapes, L.HOYER, 6, ctypes.c_void_p(vals.data_ptr()), gp,
            ctypes.c_float(0.75), stream)
    assert st == L.OK, lib.slorr_last_error()
    torch.cuda.synchronize()
    out = vals.cpu().numpy(), [g.cpu().numpy() for g in G]
    plan.close()
    return out


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_noalloc_matches_regular_entry_point(dtype):
    import torch
    import paper_2607_08754_amd._lib as L
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    sets = [([(96, 200), (300, 130), (256, 768), (7, 13)], 41),   # first call
            ([(64, 96), (33, 20)], 43)]                            # second call: a smaller set
    for shapes, seed in sets:
        v0, g0 = _run(dtype, shapes, seed, False, L)
        v1, g1 = _run(dtype, shapes, seed, True, L)
        print(f"[noalloc] {dtype} {shapes}: values {v1}", flush=True)
        assert np.all(np.isfinite(v1))
        assert np.array_equal(v1, v0)
        for a, b in zip(g1, g0):
            assert np.array_equal(a, b)
