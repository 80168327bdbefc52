"""Convenience wrapper: one DKM forward (+ optional backward) through the C ABI.

Allocates the outputs with torch on the keys' device and calls the binding;
all computation happens in the HIP library.
"""
from __future__ import annotations

import torch

from . import edkm


def as_keys(w) -> torch.Tensor:
    """fp16/bf16 weights or raw uint16/int16 patterns -> contiguous int16 view of the bits."""
    if w.element_size() != 2:
        raise ValueError("weights must be fp16, bf16 or 16-bit patterns")
    return w.contiguous().view(torch.int16)


def run(keys: torch.Tensor, c0: torch.Tensor, bits: int, tau: float, max_iter: int,
        eps: float = 0.0, grad: torch.Tensor | None = None, dense: bool = False,
        out_half: bool = False, want_counts: bool = False, want_attn: bool = False,
        check_finite: bool = False, plan: edkm.Plan | None = None,
        key_format: str = "fp16") -> dict:
    """Run init_unique + forward (+ backward when ``grad`` is given), or the dense
    path when ``dense``; returns a dict of device tensors.  ``key_format``
    ("fp16" or "bf16") says how the 16-bit patterns decode; 16-bit W~ outputs
    are of the same format."""
    dev = keys.device
    n = keys.numel()
    k = 1 << bits
    if plan is None:
        plan = edkm.Plan(n, bits, max_iter, device=dev, key_format=key_format)
    out = dict(plan=plan)
    c_out = torch.empty(k, dtype=torch.float32, device=dev)
    half = torch.bfloat16 if plan.key_format == "bf16" else torch.float16
    wt = torch.empty(n, dtype=half if out_half else torch.float32, device=dev)
    iters = torch.zeros(1, dtype=torch.int32, device=dev)
    c0 = c0.to(device=dev, dtype=torch.float32).contiguous()
    if dense:
        attn = torch.empty(n * k, dtype=torch.float32, device=dev) if want_attn else None
        edkm.forward_dense(plan, keys, tau, eps, c0, c_out, wt, out_half, iters, attn)
        if attn is not None:
            out["attn"] = attn.view(n, k)
    else:
        counts = torch.empty(edkm.NKEYS, dtype=torch.int32, device=dev) if want_counts else None
        nuniq = torch.zeros(1, dtype=torch.int32, device=dev)
        edkm.init_unique(plan, keys, counts, nuniq, check_finite)
        edkm.forward(plan, keys, tau, eps, c0, c_out, wt, out_half, iters)
        out["num_unique"] = nuniq
        if counts is not None:
            out["counts"] = counts
    out.update(c_out=c_out, w_tilde=wt, iters=iters)
    if grad is not None:
        gw = torch.empty(n, dtype=torch.float32, device=dev)
        gc = torch.empty(k, dtype=torch.float32, device=dev)
        g = grad.to(device=dev, dtype=torch.float32).contiguous()
        if dense:
            edkm.backward_dense(plan, keys, g, gw, gc)
        else:
            edkm.backward(plan, keys, g, gw, gc)
        out.update(grad_w=gw, grad_c=gc)
    return out
