"""DKM clustering of weight tensors as a differentiable torch operation.

W~ = DKM(W, C^(0)) with the uniquified forward and backward of the library
(paper Sec. 2.2): the forward runs init_unique + forward, the backward the
library's analytic backward, so a training step that uses W~ in place of W
gets dL/dW and dL/dC^(0) as autograd of the dense DKM map would give them.
dL/dW comes straight from the library in the weights' own type (fp16 or
bf16), and a 16-bit W~ takes its gradient in that type, so no cast kernels run
around the library's.
``dkm`` clusters one tensor; ``dkm_batch`` clusters a list of them (say the
seven matrices of a decoder layer) with the batched calls, one launch per step
for up to 28 matrices.  Argument marshalling only: every step runs in the HIP
library.

Each call makes its own plans (about 40 MiB of workspace per matrix through
torch's allocator), kept with the autograd graph until the backward has run,
so two clustered layers in one graph never share state.
"""
from __future__ import annotations

import torch

from . import edkm

_FORMATS = {torch.float16: "fp16", torch.bfloat16: "bf16"}


def _prepare(w, c0, max_iter):
    """Key view, plan and fp32 C^(0) of one weight tensor."""
    if not isinstance(w, torch.Tensor) or w.dtype not in _FORMATS or not w.is_cuda:
        raise TypeError("weights must be fp16 or bf16 CUDA tensors")
    k = c0.numel()
    bits = k.bit_length() - 1
    if k < 2 or k != 1 << bits or bits > 4:
        raise ValueError("C^(0) must hold 2, 4, 8 or 16 centroids")
    keys = w.detach().contiguous().view(torch.int16).view(-1)
    plan = edkm.Plan(keys.numel(), bits, int(max_iter), device=w.device, key_format=_FORMATS[w.dtype])
    c_in = c0.detach().to(device=w.device, dtype=torch.float32).contiguous()
    return keys, plan, c_in


def _grad_in(grad_wt, w):
    """dL/dW~ as the library reads it: in w's 16-bit type (the gradient of a
    16-bit W~) or as float32."""
    g = grad_wt.detach()
    if g.dtype != w.dtype:
        g = g.to(torch.float32)
    return g.contiguous().view(-1)


def _outputs(w, plan, out_half):
    c_out = torch.empty(plan.k, dtype=torch.float32, device=w.device)
    wt = torch.empty(plan.n, dtype=w.dtype if out_half else torch.float32, device=w.device)
    iters = torch.zeros(1, dtype=torch.int32, device=w.device)
    return c_out, wt, iters


class DKMFunction(torch.autograd.Function):
    """apply(w, c0, tau, max_iter, eps, out_half) -> (w_tilde, c_out, iters).

    w: fp16 or bf16 weights on the GPU (any shape; its bit patterns are the
    keys); c0: float32[2^b] starting centroids, b = 1..4; w_tilde has w's
    shape, float32 (or w's 16-bit format with out_half); c_out = C^(T) and
    iters = T are outputs without gradient."""

    @staticmethod
    def forward(ctx, w, c0, tau, max_iter, eps, out_half):
        keys, plan, c_in = _prepare(w, c0, max_iter)
        c_out, wt, iters = _outputs(w, plan, out_half)
        edkm.init_unique(plan, keys)
        edkm.forward(plan, keys, float(tau), float(eps), c_in, c_out, wt, bool(out_half), iters)
        ctx.plan = plan
        ctx.keys = keys            # the key buffer the plan was counted on
        ctx.save_for_backward(w)   # for autograd's check that w is unchanged
        ctx.mark_non_differentiable(c_out, iters)
        return wt.view(w.shape), c_out, iters

    @staticmethod
    def backward(ctx, grad_wt, grad_c_out, grad_iters):
        (w,) = ctx.saved_tensors
        plan = ctx.plan
        g = _grad_in(grad_wt, w)
        gw = torch.empty(plan.n, dtype=w.dtype, device=g.device)   # written in w's type by the library
        gc = torch.empty(plan.k, dtype=torch.float32, device=g.device)
        edkm.backward(plan, ctx.keys, g, gw, gc)
        grad_w = gw.view(w.shape) if ctx.needs_input_grad[0] else None
        grad_c0 = gc if ctx.needs_input_grad[1] else None
        return grad_w, grad_c0, None, None, None, None


class DKMBatchFunction(torch.autograd.Function):
    """apply(tau, max_iter, eps, out_half, m, w_1..w_m, c0_1..c0_m) ->
    (w_tilde_1..m, c_out_1..m, iters_1..m): DKMFunction over m tensors with
    the batched calls (same tau, eps and max_iter for all)."""

    @staticmethod
    def forward(ctx, tau, max_iter, eps, out_half, m, *tensors):
        ws, c0s = tensors[:m], tensors[m:]
        if m < 1 or len(c0s) != m:
            raise ValueError("one C^(0) per weight tensor")
        prep = [_prepare(w, c0, max_iter) for w, c0 in zip(ws, c0s)]
        keys = [p[0] for p in prep]
        plans = [p[1] for p in prep]
        outs = [_outputs(w, plan, out_half) for w, plan in zip(ws, plans)]
        c_out, wt, iters = ([o[i] for o in outs] for i in range(3))
        edkm.init_unique_batch(plans, keys)
        edkm.forward_batch(plans, keys, float(tau), float(eps), [p[2] for p in prep], c_out, wt,
                           bool(out_half), iters)
        ctx.plans, ctx.keys, ctx.m = plans, keys, m
        ctx.save_for_backward(*ws)
        ctx.mark_non_differentiable(*c_out, *iters)
        return (*[t.view(w.shape) for t, w in zip(wt, ws)], *c_out, *iters)

    @staticmethod
    def backward(ctx, *grads):
        m, plans = ctx.m, ctx.plans
        ws = ctx.saved_tensors
        g = [_grad_in(x, w) for x, w in zip(grads[:m], ws)]
        if len({x.element_size() for x in g}) > 1:        # one gradient type per batched call
            g = [x.to(torch.float32) for x in g]
        gw = [torch.empty(p.n, dtype=w.dtype, device=x.device) for p, x, w in zip(plans, g, ws)]
        gc = [torch.empty(p.k, dtype=torch.float32, device=x.device) for p, x in zip(plans, g)]
        edkm.backward_batch(plans, ctx.keys, g, gw, gc)
        need = ctx.needs_input_grad
        grad_w = [a.view(w.shape) if need[5 + i] else None for i, (a, w) in enumerate(zip(gw, ws))]
        grad_c = [a if need[5 + m + i] else None for i, a in enumerate(gc)]
        return (None, None, None, None, None, *grad_w, *grad_c)


def dkm(w, c0, tau: float = 2e-3, max_iter: int = 5, eps: float = 0.0, out_half: bool = False):
    """Clustered weights W~ (shape of w), C^(T) and T; differentiable in w and c0."""
    return DKMFunction.apply(w, c0, tau, max_iter, eps, out_half)


def dkm_batch(ws, c0s, tau: float = 2e-3, max_iter: int = 5, eps: float = 0.0, out_half: bool = False):
    """dkm over lists of weight tensors and their C^(0) with the batched calls:
    lists of W~, C^(T) and T; differentiable in every w and c0."""
    ws, c0s = list(ws), list(c0s)
    m = len(ws)
    out = DKMBatchFunction.apply(tau, max_iter, eps, out_half, m, *ws, *c0s)
    return list(out[:m]), list(out[m:2 * m]), list(out[2 * m:])
