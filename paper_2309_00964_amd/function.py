"""DKM clustering of a weight tensor as a differentiable torch operation.

W~ = DKM(W, C^(0)) with the uniquified forward and backward of the library
(paper Sec. 2.2): the forward runs init_unique + forward, the backward the
library's analytic backward, so a training step that uses W~ in place of W
gets dL/dW and dL/dC^(0) as autograd of the dense DKM map would give them.
Argument marshalling only: every step runs in the HIP library.

Each call makes its own plan (about 40 MiB of workspace through torch's
allocator), kept with the autograd graph until the backward has run, so two
clustered layers in one graph never share state.
"""
from __future__ import annotations

import torch

from . import edkm

_FORMATS = {torch.float16: "fp16", torch.bfloat16: "bf16"}


class DKMFunction(torch.autograd.Function):
    """apply(w, c0, tau, max_iter, eps, out_half) -> (w_tilde, c_out, iters).

    w: fp16 or bf16 weights on the GPU (any shape; its bit patterns are the
    keys); c0: float32[2^b] starting centroids, b = 1..4; w_tilde has w's
    shape, float32 (or w's 16-bit format with out_half); c_out = C^(T) and
    iters = T are outputs without gradient."""

    @staticmethod
    def forward(ctx, w, c0, tau, max_iter, eps, out_half):
        if w.dtype not in _FORMATS or not w.is_cuda:
            raise TypeError("w must be an fp16 or bf16 CUDA tensor")
        k = c0.numel()
        bits = k.bit_length() - 1
        if k < 2 or k != 1 << bits or bits > 4:
            raise ValueError("c0 must hold 2, 4, 8 or 16 centroids")
        wc = w.detach().contiguous()
        keys = wc.view(torch.int16).view(-1)
        n = keys.numel()
        plan = edkm.Plan(n, bits, int(max_iter), device=w.device, key_format=_FORMATS[w.dtype])
        c_in = c0.detach().to(device=w.device, dtype=torch.float32).contiguous()
        c_out = torch.empty(k, dtype=torch.float32, device=w.device)
        wt = torch.empty(n, dtype=w.dtype if out_half else torch.float32, device=w.device)
        iters = torch.zeros(1, dtype=torch.int32, device=w.device)
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
        g = grad_wt.detach().to(torch.float32).contiguous().view(-1)
        gw = torch.empty(plan.n, dtype=torch.float32, device=g.device)
        gc = torch.empty(plan.k, dtype=torch.float32, device=g.device)
        edkm.backward(plan, ctx.keys, g, gw, gc)
        grad_w = gw.view(w.shape).to(w.dtype) if ctx.needs_input_grad[0] else None
        grad_c0 = gc if ctx.needs_input_grad[1] else None
        return grad_w, grad_c0, None, None, None, None


def dkm(w, c0, tau: float = 2e-3, max_iter: int = 5, eps: float = 0.0, out_half: bool = False):
    """Clustered weights W~ (shape of w), C^(T) and T; differentiable in w and c0."""
    return DKMFunction.apply(w, c0, tau, max_iter, eps, out_half)
