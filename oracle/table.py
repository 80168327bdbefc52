"""Uniquified (table-form) DKM in fp64 numpy — a SECOND oracle.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper's Sec. 2.2 (weight uniquification, Fig. "mem_dkm:flow"): a 16-bit
weight has at most 2^16 distinct bit patterns, every weight with the same
pattern has the same attention row, so the N x k map is an attention table
with one row per distinct pattern plus an index list whose entry is the
weight's own bit pattern.  Sums over weights become sums over table rows
weighted by how many weights carry that pattern (``counts``).

This module computes exactly what ``dense`` computes, grouped by key.  In exact
arithmetic the two agree; the tests pin this module to ``dense`` (<= 1e-12
relative) before it is trusted at sizes the dense oracle cannot finish.

The decode here goes through numpy's own types (float16 for fp16 patterns, the
upper half of a float32 for bf16 ones), independently of the C oracle's
bit-level decode.
"""
from __future__ import annotations

import numpy as np

NKEYS = 1 << 16


def histogram(keys: np.ndarray) -> np.ndarray:
    """counts[u] = #{i : bits(w_i) = u} for every 16-bit pattern u (uint32)."""
    return np.bincount(np.asarray(keys, dtype=np.uint16).ravel().astype(np.int64),
                       minlength=NKEYS).astype(np.uint32)


def unique_keys(keys: np.ndarray):
    """(occupied keys ascending, inverse index) — the index list of Sec. 2.2
    compacted to ranks; ascending key order as ``np.unique`` gives it."""
    u, inv = np.unique(np.asarray(keys, dtype=np.uint16).ravel(), return_inverse=True)
    return u, inv.astype(np.uint32)


def key_values(u: np.ndarray, fmt: str = "fp16") -> np.ndarray:
    u = np.asarray(u, dtype=np.uint16)
    if fmt == "fp16":
        return u.view(np.float16).astype(np.float64)
    if fmt == "bf16":
        return (u.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    raise ValueError("fmt must be 'fp16' or 'bf16'")


def _softmax_rows(v: np.ndarray, c: np.ndarray, tau: float) -> np.ndarray:
    d = -np.abs(v[:, None] - c[None, :]) / tau
    d -= d.max(axis=1, keepdims=True)
    e = np.exp(d)
    return e / e.sum(axis=1, keepdims=True)


def forward(keys: np.ndarray, c0, tau: float, max_iter: int, eps: float = 0.0,
            counts: np.ndarray | None = None, fmt: str = "fp16") -> dict:
    """Table-form DKM forward.  Same outputs as ``dense.forward`` plus the
    per-key tables (``u``, ``n_u``, ``tab``).  ``fmt`` says how the 16-bit
    patterns decode ("fp16" or "bf16")."""
    keys = np.asarray(keys, dtype=np.uint16).ravel()
    if counts is None:
        counts = histogram(keys)
    u = np.flatnonzero(counts)
    n_u = counts[u].astype(np.float64)
    v = key_values(u, fmt)
    c0 = np.asarray(c0, dtype=np.float64).ravel()
    k = c0.size
    c_hist = np.zeros((max_iter + 1, k))
    s_hist = np.zeros((max_iter + 1, k))
    c_hist[0] = c0
    T = max_iter
    for t in range(1, max_iter + 1):
        cp = c_hist[t - 1]
        a = _softmax_rows(v, cp, tau)
        S = n_u @ a
        P = (n_u * v) @ a
        s_hist[t] = S
        c_hist[t] = np.where(S > 0, P / np.where(S > 0, S, 1.0), cp)
        if eps > 0 and np.max(np.abs(c_hist[t] - cp)) <= eps:
            T = t
            break
    aT = _softmax_rows(v, c_hist[T - 1], tau)
    tab = aT @ c_hist[T]
    tab_full = np.zeros(NKEYS)
    tab_full[u] = tab
    return dict(T=T, c_hist=c_hist, s_hist=s_hist, c_out=c_hist[T].copy(),
                w_tilde=tab_full[keys], tau=float(tau), k=k, u=u, n_u=n_u, v=v, tab=tab,
                counts=counts)


def backward(keys: np.ndarray, fwd: dict, g: np.ndarray):
    """Table-form backward of L = sum_i g_i W~_i.

    dL/dw_i = g_i * H[key_i] + R[key_i]; H, R and dL/dC^(0) are computed on the
    table from G_u = sum over weights with key u of g_i.  Returns
    (dL/dw, dL/dC^(0), extras) with extras holding G, H, R per occupied key.
    """
    keys = np.asarray(keys, dtype=np.uint16).ravel()
    g = np.asarray(g, dtype=np.float64).ravel()
    tau, T = fwd["tau"], fwd["T"]
    u, n_u, v = fwd["u"], fwd["n_u"], fwd["v"]
    c_hist, s_hist = fwd["c_hist"], fwd["s_hist"]
    G = np.bincount(keys.astype(np.int64), weights=g, minlength=NKEYS)[u]

    cT, cTm1 = c_hist[T], c_hist[T - 1]
    aT = _softmax_rows(v, cTm1, tau)
    sT = np.sign(v[:, None] - cTm1[None, :])
    tab = aT @ cT
    q = aT * (cT[None, :] - tab[:, None]) * sT
    H = -q.sum(axis=1) / tau
    gam = G @ aT
    E = (G @ q) / tau
    R = np.zeros_like(v)
    for t in range(T, 0, -1):
        ct, cp, S = c_hist[t], c_hist[t - 1], s_hist[t]
        pos = S > 0
        Ssafe = np.where(pos, S, 1.0)
        a = _softmax_rows(v, cp, tau)
        s = np.sign(v[:, None] - cp[None, :])
        al = np.where(pos[None, :], gam[None, :] * (v[:, None] - ct[None, :]) / Ssafe[None, :], 0.0)
        abar = (a * al).sum(axis=1)
        delta = a * (al - abar[:, None]) * s
        R += (a * np.where(pos, gam / Ssafe, 0.0)[None, :]).sum(axis=1) - delta.sum(axis=1) / tau
        nxt = (n_u @ delta) / tau
        if t == T:
            nxt = nxt + E
        nxt = nxt + np.where(pos, 0.0, gam)
        gam = nxt
    H_full = np.zeros(NKEYS)
    R_full = np.zeros(NKEYS)
    H_full[u] = H
    R_full[u] = R
    gw = g * H_full[keys] + R_full[keys]
    return gw, gam, dict(G=G, H=H, R=R)
