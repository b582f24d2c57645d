"""PyTorch integration of the SLORR library: argument marshalling and autograd
plumbing only; every step of the regularizer runs in libslorr.so.

  SlorrFunction    torch.autograd.Function with Listing 1's contract: forward
                   returns the per-matrix values L_i; backward returns
                   g_i dL_i/dW_i for the incoming gradients g_i. The forward
                   runs the whole iteration once and leaves the last iterate P
                   and the gradient factors in the plan's workspace (deferred
                   gradient); backward is one gradient kernel that reads g_i on
                   the device, so nothing waits on the host.
  Regularizer      a fixed list of weight parameters (conv kernels seen as
                   (C_out, C_in k_h k_w), App. C.1) with
                     loss()              values, connected to autograd (Listing 1)
                     accumulate_grad_()  App. E.3: W.grad += lambda G(W), or
                                         lambda G(W) where W has no gradient yet
                     values()            values only
                   The two gradient routes give bit-identical .grad (the
                   library rounds fl(g t) and then fl(old + fl(g t)) in both).
  DecoupledSlorr   App. E.2, Alg. 1 around a torch optimizer: the gradient of
                   the weights before the step, the optimizer's step, then
                   W <- W - eta lambda G_pre in one library kernel.
"""
from __future__ import annotations

from typing import Iterable, List, Optional

import torch

from .slorr import Plan

__all__ = ["SlorrFunction", "Regularizer", "DecoupledSlorr"]

_DT = {torch.float32: "f32", torch.bfloat16: "bf16"}


def _as_matrix(t: torch.Tensor) -> torch.Tensor:
    """2-D view of a weight: (C_out, C_in k_h k_w) for conv kernels."""
    if t.dim() < 2:
        raise ValueError("SLORR regularizes matrices; got a tensor of shape " + str(tuple(t.shape)))
    if not t.is_contiguous():
        raise ValueError("SLORR needs contiguous weights")
    return t if t.dim() == 2 else t.view(t.shape[0], -1)


class SlorrFunction(torch.autograd.Function):
    """forward(plan, *W) -> values (n,); the plan must be made with
    defer_grad=True and grad_dtype equal to the weights' dtype."""

    @staticmethod
    def forward(ctx, plan: Plan, *weights):
        vals = plan(list(weights))
        ctx.plan = plan
        ctx.generation = plan.generation
        ctx.save_for_backward(*weights)
        return vals[: plan.n].clone()

    @staticmethod
    def backward(ctx, grad_vals):
        plan: Plan = ctx.plan
        if plan.generation != ctx.generation:
            raise RuntimeError("SLORR: the plan ran another forward before this backward; its "
                               "workspace no longer holds this forward's state (use one plan per "
                               "pending backward)")
        weights = ctx.saved_tensors
        gdt = torch.bfloat16 if plan.grad_dtype == "bf16" else torch.float32
        grads = [torch.empty(w.shape, dtype=gdt, device=w.device) for w in weights]
        plan.grad(list(weights), grads, scales=grad_vals.detach().to(torch.float32).contiguous())
        return (None, *grads)


class Regularizer:
    """SLORR over a fixed list of weights (all of one dtype: float32 or bfloat16).

    kind "hoyer" (SLORR-Hoyer) or "nuclear" (SLORR-Nuc); iters, eps, ell,
    degree and coeffs as in Plan. Plans (and their workspaces) are made on
    first use.
    """

    def __init__(self, params: Iterable[torch.Tensor], kind: str = "hoyer", iters: int = 6,
                 eps: float = 0.0, ell: float = 1e-3, degree: int = 5, coeffs=None):
        self.params = list(params)
        if not self.params:
            raise ValueError("no parameters")
        dts = {p.dtype for p in self.params}
        if len(dts) != 1 or next(iter(dts)) not in _DT:
            raise ValueError("all regularized weights must share one dtype, float32 or bfloat16")
        self.dtype = _DT[next(iter(dts))]
        self.device = self.params[0].device
        self.shapes = [tuple(_as_matrix(p.detach()).shape) for p in self.params]
        self.opts = dict(kind=kind, iters=iters, eps=eps, ell=ell, degree=degree, coeffs=coeffs)
        self._plans = {}

    def plan(self, use: str) -> Plan:
        """'autograd' (deferred gradient), 'accumulate' (App. E.3) or 'values'."""
        if use not in self._plans:
            kw = dict(self.opts, dtype=self.dtype, device=self.device, grad_dtype=self.dtype)
            if use == "autograd":
                kw["defer_grad"] = True
            elif use == "accumulate":
                kw["accumulate"] = True
            elif use == "values":
                kw["values_only"] = True
            else:
                raise ValueError(use)
            self._plans[use] = Plan(self.shapes, **kw)
        return self._plans[use]

    def matrices(self, detach: bool = False) -> List[torch.Tensor]:
        return [_as_matrix(p.detach() if detach else p) for p in self.params]

    def loss(self) -> torch.Tensor:
        """Per-matrix values L_i as an autograd-connected tensor (Listing 1)."""
        return SlorrFunction.apply(self.plan("autograd"), *self.matrices())

    @torch.no_grad()
    def values(self) -> torch.Tensor:
        """Per-matrix values then their sum, no gradient."""
        return self.plan("values")(self.matrices(detach=True)).clone()

    @torch.no_grad()
    def accumulate_grad_(self, lam: float) -> torch.Tensor:
        """App. E.3: W.grad <- W.grad + lam G(W) for every weight (a zero
        gradient is created where none exists). Returns the values and sum."""
        grads = []
        for p in self.params:
            if p.grad is None:
                p.grad = torch.zeros_like(p, memory_format=torch.contiguous_format)
            if not p.grad.is_contiguous():
                raise ValueError("SLORR accumulates into contiguous .grad tensors only")
            grads.append(_as_matrix(p.grad))
        return self.plan("accumulate")(self.matrices(detach=True), grads, grad_scale=float(lam)).clone()


class DecoupledSlorr:
    """Alg. 1 (App. E.2): wraps `optimizer`; step() computes G_pre of the
    regularized weights, runs optimizer.step(), then applies
    W <- W - eta lam G_pre with eta the learning rate of each weight's group."""

    def __init__(self, optimizer: torch.optim.Optimizer, params: Iterable[torch.Tensor], lam: float,
                 **reg_kw):
        self.optimizer = optimizer
        self.lam = float(lam)
        self.reg = Regularizer(params, **reg_kw)
        self._plan = Plan(self.reg.shapes, dtype=self.reg.dtype, device=self.reg.device,
                          grad_dtype="f32", **self.reg.opts)
        self.g_pre = [torch.empty(s, dtype=torch.float32, device=self.reg.device) for s in self.reg.shapes]
        self.last_values: Optional[torch.Tensor] = None

    def _lrs(self) -> List[float]:
        out = []
        for p in self.reg.params:
            lr = None
            for grp in self.optimizer.param_groups:
                if any(q is p for q in grp["params"]):
                    lr = float(grp["lr"])
                    break
            if lr is None:
                raise ValueError("a regularized weight is not in the optimizer")
            out.append(lr)
        return out

    @torch.no_grad()
    def step(self, closure=None):
        mats = self.reg.matrices(detach=True)
        self.last_values = self._plan(mats, self.g_pre, grad_scale=1.0).clone()    # G_pre, values
        loss = self.optimizer.step(closure)
        lrs = self._lrs()
        if all(lr == lrs[0] for lr in lrs):
            self._plan.apply_update(mats, self.g_pre, step=lrs[0] * self.lam)
        else:
            steps = torch.tensor(lrs, dtype=torch.float32, device=self.reg.device)
            self._plan.apply_update(mats, self.g_pre, step=self.lam, steps=steps)
        return loss

    def zero_grad(self, set_to_none: bool = True):
        self.optimizer.zero_grad(set_to_none=set_to_none)
