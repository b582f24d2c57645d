"""GPU tests of the PyTorch integration (Listing 1, App. E.2 Alg. 1, App. E.3):
the autograd route and the accumulate (hook) route against the oracle and
against each other bit for bit, the deferred gradient against the one-call
path, the decoupled step against the oracle's Alg. 1 with AdamW, and the
decoupled update kernel against its plain definition.
"""
import numpy as np
import pytest

from oracle.pe_schedule import default_table
from oracle.slorr import fwd_bwd
from oracle.training import AdamWState, decoupled_step
from parity_util import TOL, grad_errs, to_device, value_err
from workloads import gaussian, widen

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
# ragged, tall, wide, square-ish and a conv kernel (C_out, C_in, k, k)
SHAPES = [(96, 160), (200, 72), (32, 8, 3, 3), (130, 257)]
TABLE = default_table(6)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    import paper_2607_08754_amd._lib as L
    L.lib()


def _arrays(dtype, seed):
    out = []
    for i, s in enumerate(SHAPES):
        m = (s[0], int(np.prod(s[1:])))
        out.append(gaussian(m, seed, 0.05, dtype, i))
    return out


def _params(arrs, dtype):
    import torch
    ts = to_device(arrs, dtype, DEV)
    return [torch.nn.Parameter(t.view(s)) for t, s in zip(ts, SHAPES)]


def _mat(t):
    return t.detach().reshape(t.shape[0], -1).float().cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("kind", ["hoyer", "nuclear"])
def test_autograd_matches_oracle(dtype, kind):
    """The autograd route (deferred gradient, Listing 1) against the oracle,
    with a different upstream factor per matrix."""
    import torch
    from paper_2607_08754_amd import Regularizer
    arrs = _arrays(dtype, 11)
    params = _params(arrs, dtype)
    reg = Regularizer(params, kind=kind)
    c = torch.tensor([0.5, -1.25, 2.0, 1.0], device=DEV)
    L = reg.loss()
    (L * c).sum().backward()
    torch.cuda.synchronize()
    vals = L.detach().cpu().numpy().astype(np.float64)
    for i, a in enumerate(arrs):
        ref = fwd_bwd(widen(a, dtype), kind, TABLE, g=float(c[i]))
        ve = value_err(vals[i], ref)
        gf, gm = grad_errs(_mat(params[i].grad), ref, kind, g=float(c[i]))
        print(f"[integration] autograd {dtype} {kind} matrix {i} {SHAPES[i]}: "
              f"value {ve:.2e} grad {gf:.2e} element-wise {gm:.2e}", flush=True)
        assert params[i].grad.dtype == params[i].dtype and params[i].grad.shape == params[i].shape
        assert ve <= TOL[dtype] and gf <= TOL[dtype] and gm <= TOL[dtype]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_autograd_and_accumulate_routes_are_bitwise_equal(dtype):
    """loss = task + lam sum L through autograd vs task.backward() then
    W.grad += lam G in the library (App. E.3)."""
    import torch
    from paper_2607_08754_amd import Regularizer
    arrs = _arrays(dtype, 12)
    params = _params(arrs, dtype)
    C = [torch.randn(p.shape, generator=torch.Generator().manual_seed(i)).to(DEV) for i, p in enumerate(params)]
    lam = 0.375                                   # exact in every format

    def task():
        return sum(((p.float() - c) ** 2).sum() for p, c in zip(params, C))

    reg = Regularizer(params, kind="hoyer")
    (task() + lam * reg.loss().sum()).backward()
    g_auto = [p.grad.clone() for p in params]
    for p in params:
        p.grad = None
    task().backward()
    reg.accumulate_grad_(lam)
    torch.cuda.synchronize()
    for i, p in enumerate(params):
        assert p.grad.dtype == g_auto[i].dtype
        assert torch.equal(p.grad, g_auto[i]), f"matrix {i}: max diff {(p.grad.float() - g_auto[i].float()).abs().max()}"
    # accumulate into no existing gradient: equals lam G alone
    for p in params:
        p.grad = None
    reg.accumulate_grad_(lam)
    g_only = [p.grad.clone() for p in params]
    for p in params:
        p.grad = None
    (lam * reg.loss().sum()).backward()
    for i, p in enumerate(params):
        assert torch.equal(p.grad, g_only[i])


def test_deferred_gradient_equals_one_call_path():
    import torch
    from paper_2607_08754_amd import Plan, Regularizer
    arrs = _arrays("f32", 13)
    params = _params(arrs, "f32")
    reg = Regularizer(params, kind="hoyer")
    L = reg.loss()
    L.sum().backward()
    shapes = [tuple(_mat(p).shape) for p in params]
    plan = Plan(shapes, dtype="f32", kind="hoyer", device=DEV)
    G = [torch.empty(s, dtype=torch.float32, device=DEV) for s in shapes]
    vals = plan([p.detach().view(s) for p, s in zip(params, shapes)], G)
    torch.cuda.synchronize()
    assert torch.equal(vals[: len(shapes)], L.detach())
    for p, g, s in zip(params, G, shapes):
        assert torch.equal(p.grad.view(s), g)
    # values-only route
    v2 = reg.values()
    assert torch.equal(v2[: len(shapes)], L.detach())
    # the set total: written by the gradient launch in the one-call plan and
    # by a launch of its own in the values-only plan, the same sum in the same order
    n = len(shapes)
    assert torch.equal(vals[n], v2[n])


def test_backward_after_another_forward_raises():
    from paper_2607_08754_amd import Regularizer
    params = _params(_arrays("f32", 14), "f32")
    reg = Regularizer(params, kind="hoyer")
    L1 = reg.loss()
    L2 = reg.loss()
    with pytest.raises(RuntimeError, match="another forward"):
        L1.sum().backward()
    L2.sum().backward()                          # the latest forward is still valid


def test_deferred_gradient_errors():
    import torch
    from paper_2607_08754_amd import Plan, SlorrError
    shapes = [(64, 96)]
    W = [torch.zeros(shapes[0], dtype=torch.float32, device=DEV)]
    G = [torch.zeros(shapes[0], dtype=torch.float32, device=DEV)]
    p = Plan(shapes, dtype="f32", defer_grad=True, device=DEV)
    with pytest.raises(SlorrError, match="no forward state"):
        p.grad(W, G)
    pv = Plan(shapes, dtype="f32", values_only=True, device=DEV)
    pv(W)
    with pytest.raises(SlorrError, match="values only"):
        pv.grad(W, G)


@pytest.mark.parametrize("kind", ["hoyer", "nuclear"])
def test_decoupled_step_matches_oracle(kind):
    """Alg. 1 with torch's AdamW on fp32 weights: two steps, one matrix with
    no task gradient (AdamW skips it, the SLORR term still applies)."""
    import torch
    from paper_2607_08754_amd import DecoupledSlorr
    arrs = _arrays("f32", 15)
    params = _params(arrs, "f32")
    task = [gaussian((s[0], int(np.prod(s[1:]))), 99, 0.01, "f32", i) for i, s in enumerate(SHAPES)]
    task[1] = None
    lr, lam, wd = 1e-2, 0.5, 0.05
    opt = torch.optim.AdamW(params, lr=lr, betas=(0.9, 0.999), eps=1e-8, weight_decay=wd)
    dec = DecoupledSlorr(opt, params, lam, kind=kind)
    W_ref = [widen(a, "f32") for a in arrs]
    W0 = [w.copy() for w in W_ref]
    st = [AdamWState.zeros_like(w) for w in W_ref]
    for _ in range(2):
        for p, g in zip(params, task):
            p.grad = None if g is None else torch.from_numpy(g).to(DEV).view(p.shape)
        dec.step()
        W_ref, _ = decoupled_step(W_ref, [None if g is None else g.astype(np.float64) for g in task], st,
                                  lr, lam, kind, TABLE, weight_decay=wd)
    torch.cuda.synchronize()
    for i, p in enumerate(params):
        Wg = _mat(p)
        err = np.linalg.norm(Wg - W_ref[i]) / np.linalg.norm(W_ref[i] - W0[i])
        print(f"[integration] decoupled {kind} matrix {i}: error / update size {err:.2e}", flush=True)
        assert err <= TOL["f32"]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("grad_dtype", ["f32", "bf16"])
def test_apply_update_is_its_definition(dtype, grad_dtype):
    """W <- W - s G per element: fl(w - fl(s g)), one rounding to W's type."""
    import torch
    from paper_2607_08754_amd import Plan
    shapes = [(96, 160), (200, 72), (1, 9), (130, 257)]
    plan = Plan(shapes, dtype=dtype, grad_dtype=grad_dtype, device=DEV)
    wt = torch.bfloat16 if dtype == "bf16" else torch.float32
    gt = torch.bfloat16 if grad_dtype == "bf16" else torch.float32
    gen = torch.Generator().manual_seed(5)
    W = [torch.randn(s, generator=gen).to(wt).to(DEV) for s in shapes]
    G = [torch.randn(s, generator=gen).to(gt).to(DEV) for s in shapes]
    steps = torch.tensor([0.5, 0.25, 2.0, 1.0], dtype=torch.float32, device=DEV)
    for st, sv in ((0.0625, None), (0.125, steps)):
        ref = []
        for i, (w, g) in enumerate(zip(W, G)):
            s = st if sv is None else st * float(sv[i])
            ref.append((w.float() - s * g.float()).to(wt))
        plan.apply_update(W, G, step=st, steps=sv)
        torch.cuda.synchronize()
        for i in range(len(shapes)):
            assert torch.equal(W[i], ref[i]), (i, st)
