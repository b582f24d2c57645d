"""GPU pins: closed forms and invariants the method fixes, checked on the HIP
path itself (through the C ABI), beside the oracle comparison.

  orthonormal rows   n = P phi(P^-1/2), Hoyer ratio sqrt(P) phi(P^-1/2), and a
                     Hoyer gradient that vanishes (Sec. 3 definitions; Eq.
                     SLORR_grads: the maximum of the ratio is stationary)
  diagonal           the iteration keeps a (rectangular) diagonal matrix
                     exactly diagonal: zero entries, and every off-diagonal
                     entry, of the gradient are exactly 0
  2^k scaling        with eps = 0 the value is invariant and the gradient
                     scales by 2^-k, bit for bit (Sec. 3.1, scale invariance)
  transpose          L(W^T) = L(W), grad(W^T) = grad(W)^T, bit for bit for
                     non-square W (one canonical computation for both)
  orthogonality      <W, G> = 0 for the Hoyer gradient (Sec. 3.1), here also
                     for the approximate one since n = sum(W * P) for the P
                     the gradient uses
phi is the composition of the schedule's scalar polynomials; E_T its largest
deviation from 1 on [ell, 1].
"""
import ctypes

import numpy as np
import pytest

from oracle.pe_schedule import default_table
from parity_util import TOL, compare, run_gpu, run_oracle, to_device
from workloads import f32_to_bf16_bits, gaussian, make_set, widen

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    import paper_2607_08754_amd._lib as L
    L.lib()


def _phi(x, table):
    """The scalar map of the schedule: p_T o ... o p_1 (x)."""
    x = np.asarray(x, dtype=np.float64)
    for a, b, c in np.asarray(table, dtype=np.float64):
        x = a * x + b * x ** 3 + c * x ** 5
    return x


def _store(W, dtype):
    return f32_to_bf16_bits(W.astype(np.float32)) if dtype == "bf16" else W.astype(np.float32)


def _orthonormal_rows(P, Q, seed):
    rng = np.random.default_rng([seed, P, Q])
    Z = rng.standard_normal((Q, P))
    V, R = np.linalg.qr(Z)
    return (V * np.sign(np.diag(R))[None, :]).T * 0.125        # Q x Q^T = I / 64


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_orthonormal_rows(dtype):
    table = default_table(6)
    xs = np.linspace(1e-3, 1.0, 20001)
    E = float(np.max(np.abs(1.0 - _phi(xs, table))))
    shapes = [(128, 512), (256, 768), (768, 256), (200, 600)]
    arrs = []
    for i, (m, n) in enumerate(shapes):
        Wt = _orthonormal_rows(min(m, n), max(m, n), 5 + i)
        arrs.append(_store(Wt if m <= n else Wt.T, dtype))
    tol = TOL[dtype]
    for kind in ("hoyer", "nuclear"):
        vals, grads, _ = run_gpu(arrs, dtype, kind, 6)
        refs = run_oracle(arrs, dtype, kind, 6)
        compare(vals, grads, refs, kind, dtype, label=f"orthonormal {dtype}", stationary=(kind == "hoyer"))
        for i, (m, n) in enumerate(shapes):
            P = min(m, n)
            c = _phi(P ** -0.5, table)                            # sigma / ||W||_F = P^-1/2
            if kind == "hoyer":
                r = np.sqrt(vals[i])
                assert abs(r - np.sqrt(P) * c) <= tol * np.sqrt(P) * c, (i, r, np.sqrt(P) * c)
                assert abs(r - np.sqrt(P)) <= (E + tol) * np.sqrt(P)
                # the gradient vanishes: relative to its first term s1 P
                s1 = 2.0 * refs[i].n_hat / refs[i].f_eps ** 2
                assert np.linalg.norm(grads[i]) <= tol * s1 * np.linalg.norm(refs[i].polar), i
            else:
                nuc = P * 0.125                                   # ||W||_* = P sigma, sigma = 1/8
                assert abs(vals[i] - nuc * c) <= tol * nuc * c, (i, vals[i], nuc * c)
                assert abs(vals[i] - nuc) <= (E + tol) * nuc
        print(f"[pins] orthonormal rows {dtype} {kind}: values {vals[:len(shapes)]}", flush=True)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_diagonal_stays_diagonal(dtype):
    shapes = [(96, 200), (200, 96), (130, 130), (64, 64)]
    arrs = []
    for i, (m, n) in enumerate(shapes):
        k = min(m, n)
        rng = np.random.default_rng([77, i])
        d = rng.uniform(0.01, 0.5, k) * rng.choice([-1.0, 1.0], k)
        d[rng.choice(k, k // 5, replace=False)] = 0.0              # zero singular values
        W = np.zeros((m, n))
        W[np.arange(k), np.arange(k)] = d
        arrs.append(_store(W, dtype))
    for kind in ("hoyer", "nuclear"):
        vals, grads, _ = run_gpu(arrs, dtype, kind, 6, g=0.75)
        refs = run_oracle(arrs, dtype, kind, 6, g=0.75)
        compare(vals, grads, refs, kind, dtype, g=0.75, label=f"diagonal {dtype}")
        for i, (m, n) in enumerate(shapes):
            k = min(m, n)
            Wd = widen(arrs[i], dtype)
            off = np.ones((m, n), bool)
            off[np.arange(k), np.arange(k)] = False
            assert np.all(grads[i][off] == 0.0), (i, "off-diagonal gradient entries")
            zero = np.zeros((m, n), bool)
            zero[np.arange(k), np.arange(k)] = Wd[np.arange(k), np.arange(k)] == 0.0
            assert np.all(grads[i][zero] == 0.0), (i, "gradient at zero diagonal entries")
            assert np.any(zero)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_power_of_two_scaling_is_bitwise(dtype):
    shapes = [(96, 200), (200, 96), (130, 130), (7, 300)]
    arrs = [gaussian(s, seed=91, std=0.05, dtype=dtype, index=i) for i, s in enumerate(shapes)]
    for kind in ("hoyer", "nuclear"):
        v0, g0, _ = run_gpu(arrs, dtype, kind, 6, eps=0.0)
        for k in (3, -2):
            sc = [_store(widen(a, dtype) * 2.0 ** k, dtype) for a in arrs]
            v1, g1, _ = run_gpu(sc, dtype, kind, 6, eps=0.0)
            if kind == "hoyer":
                assert np.array_equal(v1, v0), (k, v1 - v0)
                for a, b in zip(g1, g0):
                    assert np.array_equal(a, b * 2.0 ** -k), k          # grad(2^k W) = grad(W) / 2^k
            else:
                assert np.array_equal(v1[:len(shapes)], v0[:len(shapes)] * 2.0 ** k), k   # homogeneous
                for a, b in zip(g1, g0):
                    assert np.array_equal(a, b), k                        # P is scale free
        print(f"[pins] 2^k scaling {dtype} {kind}: bitwise", flush=True)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_transpose_is_bitwise(dtype):
    shapes = [(96, 200), (300, 130), (7, 300), (256, 768)]
    arrs = [gaussian(s, seed=93, std=0.05, dtype=dtype, index=i) for i, s in enumerate(shapes)]
    tr = [np.ascontiguousarray(a.T) for a in arrs]
    for kind in ("hoyer", "nuclear"):
        v0, g0, _ = run_gpu(arrs, dtype, kind, 6, eps=1e-4, g=0.5)
        v1, g1, _ = run_gpu(tr, dtype, kind, 6, eps=1e-4, g=0.5)
        assert np.array_equal(v0, v1)
        for a, b in zip(g0, g1):
            assert np.array_equal(a, b.T)
    # a square matrix and its transpose take different canonical operands:
    # equal within the tolerance
    sq = [gaussian((200, 200), seed=95, std=0.05, dtype=dtype)]
    v0, g0, _ = run_gpu(sq, dtype, "hoyer", 6)
    v1, g1, _ = run_gpu([np.ascontiguousarray(sq[0].T)], dtype, "hoyer", 6)
    assert abs(v0[0] - v1[0]) <= TOL[dtype] * abs(v0[0])
    assert np.linalg.norm(g0[0] - g1[0].T) <= TOL[dtype] * np.linalg.norm(g0[0])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_gradient_orthogonal_to_weights(dtype):
    """|<W, G>| / (||W|| ||G||) at the rounding level of the gradient's fp32
    arithmetic (1e-6), for the ViT-B/16 shapes (the bench set's first block)
    and a ragged set, Hoyer, eps = 0."""
    arrs = make_set("vit_b16", 0, indices=range(4)) if dtype == "bf16" else \
        [gaussian(s, seed=97, std=0.05, dtype="f32", index=i) for i, s in enumerate([(768, 2304), (768, 768)])]
    arrs += [gaussian(s, seed=99, std=0.05, dtype=dtype, index=i) for i, s in enumerate([(96, 200), (300, 130)])]
    vals, grads, _ = run_gpu(arrs, dtype, "hoyer", 6, eps=0.0)
    worst = 0.0
    for a, G in zip(arrs, grads):
        W = widen(a, dtype)
        c = abs(np.sum(W * G)) / (np.linalg.norm(W) * np.linalg.norm(G))
        worst = max(worst, c)
    print(f"[pins] <W, G> / (|W| |G|) {dtype}: {worst:.2e}", flush=True)
    assert worst <= 1e-6


def test_null_plan_uses_the_plan_cache():
    """slorr_reg_fwd_bwd(NULL, ...) through the C ABI: the internal plan cache
    (slorr_cache_config dtype and options) gives bitwise the result of an
    explicit plan with the same options; a second call reuses the entry; the
    cache is released by slorr_cache_clear."""
    import torch
    import paper_2607_08754_amd._lib as L
    from paper_2607_08754_amd import Plan
    lib = L.lib()
    shapes = [(96, 200), (300, 130)]
    arrs = [gaussian(s, seed=101, std=0.05, dtype="bf16", index=i) for i, s in enumerate(shapes)]
    W = to_device(arrs, "bf16", "cuda:0")
    ref = Plan(shapes, dtype="bf16", kind="nuclear", iters=5, eps=1e-4, device="cuda:0")
    G0 = [torch.empty(s, dtype=torch.float32, device="cuda:0") for s in shapes]
    v0 = ref(W, G0, grad_scale=0.5).cpu().numpy()
    torch.cuda.synchronize()
    o = L.Options()
    lib.slorr_default_options(ctypes.byref(o))
    o.eps = 1e-4
    lib.slorr_cache_config(L.BF16, ctypes.byref(o))
    c_shapes = (L.Shape * 2)(*[L.Shape(r, c) for r, c in shapes])
    wp = (ctypes.c_void_p * 2)(*[w.data_ptr() for w in W])
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    for rep in range(2):
        G1 = [torch.full(s, float("nan"), dtype=torch.float32, device="cuda:0") for s in shapes]
        v1 = torch.empty(3, dtype=torch.float32, device="cuda:0")
        gp = (ctypes.c_void_p * 2)(*[g.data_ptr() for g in G1])
        st = lib.slorr_reg_fwd_bwd(None, 2, wp, c_shapes, L.NUCLEAR, 5, ctypes.c_void_p(v1.data_ptr()), gp,
                                   ctypes.c_float(0.5), stream)
        assert st == L.OK, lib.slorr_last_error()
        torch.cuda.synchronize()
        assert np.array_equal(v1.cpu().numpy(), v0), rep
        for a, b in zip(G1, G0):
            assert torch.equal(a, b), rep
    lib.slorr_cache_config(L.F32, None)
    assert lib.slorr_cache_clear() == L.OK


def test_large_set_matches_subset_bitwise():
    """A matrix's results do not depend on the rest of the set when every
    launch uses the same kernel configuration: 17 matrices of 4096 x 16384
    (17408 update tiles, more than 64 per block of the persistent update
    kernel, so each block reloads its tile table) against the first 4 alone
    (4096 tiles), both with 256-tiles in every GEMM launch; values and
    gradients bit for bit. Weights are drawn on the device (no oracle)."""
    import torch
    from paper_2607_08754_amd import Plan
    shape = (4096, 16384)
    gen = torch.Generator(device="cuda:0")
    gen.manual_seed(1234)
    W = [(torch.randn(shape, generator=gen, device="cuda:0") * 0.02).to(torch.bfloat16) for _ in range(17)]
    out, edges = {}, {}
    for n in (17, 4):
        plan = Plan([shape] * n, dtype="bf16", kind="hoyer", iters=6, eps=1e-4, device="cuda:0")
        edges[n] = [(op, te) for op, _, te in plan.launches()]
        G = [torch.empty(shape, dtype=torch.float32, device="cuda:0") for _ in range(4)]
        G += [torch.empty(shape, dtype=torch.float32, device="cuda:0") for _ in range(n - 4)]
        vals = plan(W[:n], G)
        torch.cuda.synchronize()
        out[n] = (vals[:4].cpu(), G[:4])
        plan.close()
        print(f"[pins] 4096x16384 set of {n}: values {out[n][0].tolist()}", flush=True)
    assert edges[17] == edges[4] and all(te == 256 for op, te in edges[4] if te), edges[4]
    assert torch.equal(out[17][0], out[4][0])
    for a, b in zip(out[17][1], out[4][1]):
        assert torch.equal(a, b)
