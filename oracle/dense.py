"""ctypes wrapper around the fp64 dense DKM oracle (``dkm_dense.c``).

TEST INFRASTRUCTURE ONLY (see the package docstring).  The shared object is
built next to the source with gcc; if it is missing it is built on first use.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "dkm_dense.c")
_LIB = os.path.join(_HERE, "libdkm_oracle.so")

_lib = None


def build(force: bool = False) -> str:
    """Compile ``dkm_dense.c`` into ``libdkm_oracle.so`` (gcc, OpenMP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(build())
        P = ctypes.c_void_p
        i64, i32, f64 = ctypes.c_int64, ctypes.c_int, ctypes.c_double
        lib.dkm_fp16_value.argtypes = [ctypes.c_uint16]
        lib.dkm_fp16_value.restype = f64
        lib.dkm_decode_fp16.argtypes = [P, i64, P]
        lib.dkm_decode_fp16.restype = None
        lib.dkm_bf16_value.argtypes = [ctypes.c_uint16]
        lib.dkm_bf16_value.restype = f64
        lib.dkm_decode_bf16.argtypes = [P, i64, P]
        lib.dkm_decode_bf16.restype = None
        lib.dkm_threads.argtypes = []
        lib.dkm_threads.restype = i32
        lib.dkm_set_threads.argtypes = [i32]
        lib.dkm_set_threads.restype = None
        for name in ("dkm_dense_forward", "dkm_dense_forward_f64"):
            fn = getattr(lib, name)
            fn.argtypes = [P, i64, i32, f64, i32, f64, P, P, P, P, P]
            fn.restype = i32
        for name in ("dkm_dense_backward", "dkm_dense_backward_f64"):
            fn = getattr(lib, name)
            fn.argtypes = [P, i64, i32, f64, i32, P, P, P, P, P]
            fn.restype = i32
        _lib = lib
    return _lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def threads() -> int:
    """OpenMP threads the oracle runs on."""
    return int(_load().dkm_threads())


def set_threads(n: int) -> None:
    """OpenMP threads for later calls (results do not depend on it)."""
    _load().dkm_set_threads(int(n))


def fp16_value(h: int) -> float:
    """Real value of one fp16 bit pattern (IEEE 754 binary16 definition)."""
    return float(_load().dkm_fp16_value(int(h) & 0xFFFF))


def decode_fp16(keys: np.ndarray) -> np.ndarray:
    keys = np.ascontiguousarray(keys, dtype=np.uint16)
    out = np.empty(keys.shape, dtype=np.float64)
    _load().dkm_decode_fp16(_ptr(keys), keys.size, _ptr(out))
    return out


def bf16_value(h: int) -> float:
    """Real value of one bfloat16 bit pattern (by the format's definition)."""
    return float(_load().dkm_bf16_value(int(h) & 0xFFFF))


def decode_bf16(keys: np.ndarray) -> np.ndarray:
    keys = np.ascontiguousarray(keys, dtype=np.uint16)
    out = np.empty(keys.shape, dtype=np.float64)
    _load().dkm_decode_bf16(_ptr(keys), keys.size, _ptr(out))
    return out


def _values(x: np.ndarray, fmt: str):
    """(array, keyed?) for the C entry points: fp16 patterns go to the keyed
    entry points, bf16 patterns are decoded here, values pass through."""
    if x.dtype == np.uint16:
        if fmt == "fp16":
            return np.ascontiguousarray(x).ravel(), True
        if fmt == "bf16":
            return decode_bf16(x).ravel(), False
        raise ValueError("fmt must be 'fp16' or 'bf16'")
    return np.ascontiguousarray(x, dtype=np.float64).ravel(), False


def forward(x: np.ndarray, c0, tau: float, max_iter: int, eps: float = 0.0,
            want_attn: bool = False, fmt: str = "fp16") -> dict:
    """Dense DKM forward.

    ``x`` is either raw 16-bit patterns (uint16; fp16 or, with ``fmt="bf16"``,
    bfloat16) or real values (float64; used by the finite-difference tests).
    Returns a dict with ``T`` (iterations executed), ``c_hist`` ((max_iter+1) x
    k; rows 0..T valid), ``s_hist``, ``c_out`` (= C^(T)), ``w_tilde`` (N) and
    optionally ``attn`` (A^(T), N x k).
    """
    lib = _load()
    c0 = np.ascontiguousarray(c0, dtype=np.float64).ravel()
    k = c0.size
    xs, keyed = _values(x, fmt)
    fn = lib.dkm_dense_forward if keyed else lib.dkm_dense_forward_f64
    n = xs.size
    c_hist = np.zeros((max_iter + 1, k))
    s_hist = np.zeros((max_iter + 1, k))
    w = np.empty(n)
    attn = np.empty((n, k)) if want_attn else None
    T = fn(_ptr(xs), n, k, float(tau), int(max_iter), float(eps), _ptr(c0), _ptr(c_hist),
           _ptr(s_hist), _ptr(w), _ptr(attn) if want_attn else None)
    if T < 1:
        raise ValueError("dense oracle rejected its arguments (status %d)" % T)
    out = dict(T=T, c_hist=c_hist, s_hist=s_hist, c_out=c_hist[T].copy(), w_tilde=w,
               tau=float(tau), k=k, fmt=fmt)
    if want_attn:
        out["attn"] = attn
    return out


def backward(x: np.ndarray, fwd: dict, g: np.ndarray):
    """Dense DKM backward of L = sum_i g_i W~_i.  Returns (dL/dw, dL/dC^(0))."""
    lib = _load()
    xs, keyed = _values(x, fwd.get("fmt", "fp16"))
    fn = lib.dkm_dense_backward if keyed else lib.dkm_dense_backward_f64
    n = xs.size
    gg = np.ascontiguousarray(g, dtype=np.float64).ravel()
    assert gg.size == n
    k = fwd["k"]
    gw = np.empty(n)
    gc = np.empty(k)
    r = fn(_ptr(xs), n, k, fwd["tau"], fwd["T"], _ptr(fwd["c_hist"]), _ptr(fwd["s_hist"]),
           _ptr(gg), _ptr(gw), _ptr(gc))
    if r != 0:
        raise ValueError("dense oracle backward failed (status %d)" % r)
    return gw, gc
