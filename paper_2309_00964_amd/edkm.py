"""Python binding of the C-ABI library ``libedkm.so`` (see ``include/edkm.h``).

Argument marshalling only: tensors become device pointers and the current HIP
stream; every step of the computation runs in the library's HIP kernels.  The
functions keep the C names without the ``edkm_`` prefix.  Importing this module
loads the library and raises ``ImportError`` if it has not been built (run
``__graft_entry__.build()``); there is no fallback.

Weights are passed as 16-bit patterns of the plan's format (fp16 or bf16): any
contiguous 2-byte device tensor (the weights themselves, or ``int16`` views).
Every tensor is checked here to be a contiguous device tensor with the element
size and at least the element count the kernels access through it (the C ABI
takes raw pointers and cannot check sizes).
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
# EDKM_LIBRARY may name another build of the same sources (the block-timeline
# diagnostics build, libedkm_stamps.so); by default the product library.
LIB_PATH = os.environ.get("EDKM_LIBRARY") or os.path.join(_HERE, "libedkm.so")

if not os.path.exists(LIB_PATH):
    raise ImportError("%s is not built; run __graft_entry__.build()" % LIB_PATH)

# torch brings its own HIP runtime (SONAME libamdhip64.so.7, loaded under the
# name libamdhip64.so).  It must be in the process before libedkm.so is loaded,
# so that libedkm.so binds to that same runtime instead of mapping a second one
# from /opt/rocm, which would not see the device.
import torch  # noqa: E402,F401

_lib = ctypes.CDLL(LIB_PATH)


def _hip_runtimes():
    try:
        with open("/proc/self/maps") as f:
            return sorted({line.split()[-1] for line in f if "libamdhip64" in line})
    except OSError:
        return []


if len(_hip_runtimes()) > 1:
    raise ImportError("two HIP runtimes are mapped in this process (%s); import torch before "
                      "loading libedkm.so" % ", ".join(_hip_runtimes()))

OK = 0
ERR_ARG = -1
ERR_NONFINITE = -2
ERR_WORKSPACE = -3
ERR_STATE = -4
ERR_HIP = -5
NKEYS = 65536
PASS_HIST, PASS_GATHER_WT, PASS_KEYED_GRAD, PASS_GATHER_GRAD = 0, 1, 2, 3
PASS_DENSE_ITER, PASS_DENSE_BITER, PASS_PALETTIZE, PASS_INVERSE = 4, 5, 6, 7
KEYS_FP16, KEYS_BF16 = 0, 1
LAUNCH_GROUP = 28          # EDKM_LAUNCH_GROUP: matrices per launch in the batched calls
KEYED_AUTO, KEYED_I32, KEYED_U64 = -1, 0, 1
KEY_FORMATS = {"fp16": KEYS_FP16, "bf16": KEYS_BF16}


class EdkmError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str = ""):
        self.status = status
        super().__init__("%s: %s (%d)%s" % (where, status_str(status), status,
                                            (" — " + detail) if detail else ""))


class edkm_plan(ctypes.Structure):
    _fields_ = [("opaque", ctypes.c_uint64 * 32)]


_P = ctypes.c_void_p
_PP = ctypes.POINTER(ctypes.c_void_p)
_i32, _u64, _f32, _sz = ctypes.c_int, ctypes.c_uint64, ctypes.c_float, ctypes.c_size_t
_PLAN = ctypes.POINTER(edkm_plan)

_SIGS = {
    "edkm_workspace_bytes": (_sz, [_u64, _i32, _i32]),
    "edkm_plan_init": (_i32, [_PLAN, _u64, _i32, _i32, _P, _sz]),
    "edkm_plan_init_ex": (_i32, [_PLAN, _u64, _i32, _i32, _i32, _P, _sz]),
    "edkm_plan_set_keyed_mode": (_i32, [_PLAN, _i32]),
    "edkm_palettize": (_i32, [_PLAN, _P, _P, _P, _P]),
    "edkm_palettize_batch": (_i32, [_i32, _PP, _PP, _PP, _PP, _P]),
    "edkm_palettize_noalloc": (_i32, [_P, _u64, _i32, _i32, _P, _P, _P]),
    "edkm_unique_inverse": (_i32, [_PLAN, _P, _P, _P, _P]),
    "edkm_unique_inverse_batch": (_i32, [_i32, _PP, _PP, _PP, _PP, _P]),
    "edkm_init_unique": (_i32, [_PLAN, _P, _P, _P, _i32, _P]),
    "edkm_forward": (_i32, [_PLAN, _P, _f32, _f32, _P, _P, _P, _i32, _P, _P]),
    "edkm_backward": (_i32, [_PLAN, _P, _P, _P, _P, _P]),
    "edkm_backward_ex": (_i32, [_PLAN, _P, _P, _P, _P, _i32, _P]),
    "edkm_init_unique_batch": (_i32, [_i32, _PP, _PP, _PP, _PP, _i32, _P]),
    "edkm_forward_batch": (_i32, [_i32, _PP, _PP, _f32, _f32, _PP, _PP, _PP, _i32, _PP, _P]),
    "edkm_backward_batch": (_i32, [_i32, _PP, _PP, _PP, _PP, _PP, _P]),
    "edkm_backward_batch_ex": (_i32, [_i32, _PP, _PP, _PP, _PP, _PP, _i32, _P]),
    "edkm_forward_dense": (_i32, [_PLAN, _P, _f32, _f32, _P, _P, _P, _i32, _P, _P, _P]),
    "edkm_backward_dense": (_i32, [_PLAN, _P, _P, _P, _P, _P]),
    "edkm_plan_set_pass_events": (_i32, [_PLAN, _i32, _P, _P]),
    "edkm_plan_hip_error": (_i32, [_PLAN, ctypes.POINTER(_i32), ctypes.POINTER(ctypes.c_char_p),
                                   ctypes.POINTER(ctypes.c_char_p)]),
    "edkm_status_str": (ctypes.c_char_p, [_i32]),
}
for _name, (_res, _args) in _SIGS.items():
    _fn = getattr(_lib, _name)
    _fn.restype = _res
    _fn.argtypes = _args

EXPORTS = tuple(_SIGS)


def status_str(status: int) -> str:
    return _lib.edkm_status_str(int(status)).decode()


def plan_hip_error(plan) -> tuple:
    """(HIP error code, failing step, HIP description) of the last EDKM_ERR_HIP on a plan."""
    code = _i32(0)
    step = ctypes.c_char_p()
    msg = ctypes.c_char_p()
    _lib.edkm_plan_hip_error(plan.ref, ctypes.byref(code), ctypes.byref(step), ctypes.byref(msg))
    return code.value, (step.value or b"").decode(), (msg.value or b"").decode()


def _check(status: int, where: str, plans=()) -> None:
    if status != OK:
        detail = ""
        if status == ERR_HIP:
            for p in plans:
                code, step, msg = plan_hip_error(p)
                if code:
                    detail = "%s failed with hipError %d (%s)" % (step, code, msg)
                    break
        raise EdkmError(status, where, detail)


def _ptr(t, nbytes_elem=None, name="tensor", count=None):
    """Device pointer of a contiguous tensor (None -> NULL) holding at least
    `count` elements: the kernels read and write that many through it."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if nbytes_elem is not None and t.element_size() != nbytes_elem:
        raise ValueError("%s must have %d-byte elements" % (name, nbytes_elem))
    if count is not None and t.numel() < count:
        raise ValueError("%s has %d elements, %d needed" % (name, t.numel(), count))
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def workspace_bytes(n: int, bits: int, max_iter: int) -> int:
    return int(_lib.edkm_workspace_bytes(int(n), int(bits), int(max_iter)))


class Plan:
    """An ``edkm_plan`` plus its device workspace (allocated through torch)."""

    def __init__(self, n: int, bits: int, max_iter: int, device="cuda", workspace=None,
                 key_format: str = "fp16"):
        import torch
        self.n, self.bits, self.k, self.max_iter = int(n), int(bits), 1 << int(bits), int(max_iter)
        if key_format not in KEY_FORMATS:
            raise EdkmError(ERR_ARG, "plan_init", "key_format must be one of %s" % sorted(KEY_FORMATS))
        self.key_format = key_format
        nbytes = workspace_bytes(n, bits, max_iter)
        if nbytes == 0:
            raise EdkmError(ERR_ARG, "workspace_bytes")
        if workspace is None:
            workspace = torch.empty(nbytes, dtype=torch.uint8, device=device)
        self.workspace = workspace
        self.plan = edkm_plan()
        _check(_lib.edkm_plan_init_ex(ctypes.byref(self.plan), self.n, self.bits, self.max_iter,
                                      KEY_FORMATS[key_format], _ptr(workspace),
                                      workspace.numel() * workspace.element_size()),
               "plan_init")

    @property
    def ref(self):
        return ctypes.byref(self.plan)


def palettize(plan: Plan, w_bits, lut, indices_out, stream=None) -> None:
    """Packed b-bit nearest-entry indices of every weight against ``lut``
    (device float[k]); ``indices_out`` holds ceil(n b / 8) bytes."""
    need = (plan.n * plan.bits + 7) // 8
    if indices_out.numel() * indices_out.element_size() < need:
        raise EdkmError(ERR_ARG, "palettize", "indices_out needs %d bytes" % need)
    _check(_lib.edkm_palettize(plan.ref, _ptr(w_bits, 2, "w_bits", plan.n), _ptr(lut, 4, "lut", plan.k),
                               _ptr(indices_out, 1),
                               _stream(stream)), "palettize", (plan,))


def palettize_noalloc(w_bits, n: int, bits: int, lut, indices_out, key_format: str = "fp16",
                      stream=None) -> None:
    """palettize without a plan or workspace: the library keeps the per-pattern
    table in its own device array (one per GPU; calls on one GPU must not
    overlap).  ``indices_out`` holds ceil(n b / 8) bytes."""
    if key_format not in KEY_FORMATS:
        raise EdkmError(ERR_ARG, "palettize_noalloc", "key_format must be one of %s" % sorted(KEY_FORMATS))
    n, bits = int(n), int(bits)
    if not 1 <= bits <= 4:
        raise EdkmError(ERR_ARG, "palettize_noalloc", "bits must be 1..4")
    _check(_lib.edkm_palettize_noalloc(_ptr(w_bits, 2, "w_bits", n), n, bits, KEY_FORMATS[key_format],
                                       _ptr(lut, 4, "lut", 1 << bits),
                                       _ptr(indices_out, 1, "indices_out", (n * bits + 7) // 8),
                                       _stream(stream)), "palettize_noalloc")


def unique_inverse(plan: Plan, w_bits, unique_out=None, inverse_out=None, stream=None) -> None:
    """The uniquification's two lists, ascending by 16-bit key (numpy.unique's
    order): the distinct patterns into ``unique_out`` (16-bit elements, room
    for 65,536; the first num_unique are written) and each weight's index
    among them into ``inverse_out`` (16-bit, n).  After init_unique on the
    same keys; at least one output."""
    _check(_lib.edkm_unique_inverse(plan.ref, _ptr(w_bits, 2, "w_bits", plan.n),
                                    _ptr(unique_out, 2, "unique_out", NKEYS),
                                    _ptr(inverse_out, 2, "inverse_out", plan.n), _stream(stream)),
           "unique_inverse", (plan,))


def plan_set_keyed_mode(plan: Plan, mode: int) -> None:
    """KEYED_AUTO (default), KEYED_I32 or KEYED_U64; effective at the next init_unique."""
    _check(_lib.edkm_plan_set_keyed_mode(plan.ref, int(mode)), "plan_set_keyed_mode", (plan,))


def plan_set_pass_events(plan: Plan, pass_id: int, start, stop) -> None:
    """Record raw hipEvent_t handles (ints, or None to clear) around an N-sized pass."""
    _check(_lib.edkm_plan_set_pass_events(plan.ref, int(pass_id), start, stop), "plan_set_pass_events")


def plan_init(n: int, bits: int, max_iter: int, device="cuda") -> Plan:
    return Plan(n, bits, max_iter, device)


def init_unique(plan: Plan, w_bits, counts_out=None, num_unique_out=None, check_finite=False,
                stream=None) -> None:
    _check(_lib.edkm_init_unique(plan.ref, _ptr(w_bits, 2, "w_bits", plan.n),
                                 _ptr(counts_out, 4, "counts_out", NKEYS),
                                 _ptr(num_unique_out, 4, "num_unique_out", 1), int(bool(check_finite)),
                                 _stream(stream)),
           "init_unique", (plan,))


def forward(plan: Plan, w_bits, tau: float, eps: float, c_in, c_out, w_tilde, out_half=False,
            iters_out=None, stream=None) -> None:
    _check(_lib.edkm_forward(plan.ref, _ptr(w_bits, 2, "w_bits", plan.n), float(tau), float(eps),
                             _ptr(c_in, 4, "c_in", plan.k), _ptr(c_out, 4, "c_out", plan.k),
                             _ptr(w_tilde, 2 if out_half else 4, "w_tilde", plan.n),
                             int(bool(out_half)), _ptr(iters_out, 4, "iters_out", 1), _stream(stream)),
           "forward", (plan,))


GRAD_IN_HALF, GRAD_OUT_HALF = 1, 2


def _grad_flags(grad_w_tilde, grad_w):
    """edkm_backward_ex flags from the gradient arrays' element sizes: 2-byte
    elements are 16-bit floats of the plan's weight format, 4-byte ones float."""
    f = 0
    for t, bit, name in ((grad_w_tilde, GRAD_IN_HALF, "grad_w_tilde"), (grad_w, GRAD_OUT_HALF, "grad_w")):
        if t.element_size() == 2:
            f |= bit
        elif t.element_size() != 4:
            raise ValueError("%s must have 2- or 4-byte elements" % name)
    return f


def backward(plan: Plan, w_bits, grad_w_tilde, grad_w, grad_c, stream=None) -> None:
    """dL/dw and dL/dC^(0); grad_w_tilde and grad_w may each be float32 or
    16-bit (the plan's weight format), chosen by their element size."""
    f = _grad_flags(grad_w_tilde, grad_w)
    _check(_lib.edkm_backward_ex(plan.ref, _ptr(w_bits, 2, "w_bits", plan.n),
                                 _ptr(grad_w_tilde, grad_w_tilde.element_size(), "grad_w_tilde", plan.n),
                                 _ptr(grad_w, grad_w.element_size(), "grad_w", plan.n),
                                 _ptr(grad_c, 4, "grad_c", plan.k), f, _stream(stream)),
           "backward", (plan,))


def forward_dense(plan: Plan, w_bits, tau: float, eps: float, c_in, c_out, w_tilde,
                  out_half=False, iters_out=None, attn_out=None, stream=None) -> None:
    _check(_lib.edkm_forward_dense(plan.ref, _ptr(w_bits, 2, "w_bits", plan.n), float(tau), float(eps),
                                   _ptr(c_in, 4, "c_in", plan.k), _ptr(c_out, 4, "c_out", plan.k),
                                   _ptr(w_tilde, 2 if out_half else 4, "w_tilde", plan.n),
                                   int(bool(out_half)), _ptr(iters_out, 4, "iters_out", 1),
                                   _ptr(attn_out, 4, "attn_out", plan.n * plan.k), _stream(stream)),
           "forward_dense", (plan,))


def backward_dense(plan: Plan, w_bits, grad_w_tilde, grad_w, grad_c, stream=None) -> None:
    _check(_lib.edkm_backward_dense(plan.ref, _ptr(w_bits, 2, "w_bits", plan.n),
                                    _ptr(grad_w_tilde, 4, "grad_w_tilde", plan.n),
                                    _ptr(grad_w, 4, "grad_w", plan.n), _ptr(grad_c, 4, "grad_c", plan.k),
                                    _stream(stream)),
           "backward_dense", (plan,))


def _parr(items, esize=None, name="tensor", counts=None):
    """Host array of device pointers; counts[i] = elements items[i] must hold."""
    counts = counts or [None] * len(items)
    arr = (ctypes.c_void_p * len(items))(*[_ptr(t, esize, "%s[%d]" % (name, i), c)
                                             for i, (t, c) in enumerate(zip(items, counts))])
    return ctypes.cast(arr, _PP), arr


def _plans(plans):
    arr = (ctypes.c_void_p * len(plans))(*[ctypes.addressof(p.plan) for p in plans])
    return ctypes.cast(arr, _PP), arr


def _same_len(where, plans, **lists):
    """Every per-matrix list of a batched call has one entry per plan (the C
    side reads `count` entries of each host array)."""
    for name, items in lists.items():
        if items is not None and len(items) != len(plans):
            raise EdkmError(ERR_ARG, where, "%s has %d entries for %d plans" % (name, len(items), len(plans)))


def init_unique_batch(plans, w_bits, counts_out=None, num_unique_out=None, check_finite=False,
                      stream=None) -> None:
    _same_len("init_unique_batch", plans, w_bits=w_bits, counts_out=counts_out, num_unique_out=num_unique_out)
    n = len(plans)
    pp, _a = _plans(plans)
    ns, ks = [p.n for p in plans], [p.k for p in plans]
    kk, _b = _parr(w_bits, 2, "w_bits", ns)
    co, _c = _parr(counts_out, 4, "counts_out", [NKEYS] * n) if counts_out is not None else (None, None)
    nu, _d = _parr(num_unique_out, 4, "num_unique_out", [1] * n) if num_unique_out is not None else (None, None)
    _check(_lib.edkm_init_unique_batch(n, pp, kk, co, nu, int(bool(check_finite)), _stream(stream)),
           "init_unique_batch", plans)


def forward_batch(plans, w_bits, tau, eps, c_in, c_out, w_tilde, out_half=False, iters_out=None,
                  stream=None) -> None:
    _same_len("forward_batch", plans, w_bits=w_bits, c_in=c_in, c_out=c_out, w_tilde=w_tilde, iters_out=iters_out)
    n = len(plans)
    pp, _a = _plans(plans)
    ns, ks = [p.n for p in plans], [p.k for p in plans]
    kk, _b = _parr(w_bits, 2, "w_bits", ns)
    ci, _c = _parr(c_in, 4, "c_in", ks)
    co, _d = _parr(c_out, 4, "c_out", ks)
    wt, _e = _parr(w_tilde, 2 if out_half else 4, "w_tilde", ns)
    it, _f = _parr(iters_out, 4, "iters_out", [1] * n) if iters_out is not None else (None, None)
    _check(_lib.edkm_forward_batch(n, pp, kk, float(tau), float(eps), ci, co, wt,
                                   int(bool(out_half)), it, _stream(stream)),
           "forward_batch", plans)


def backward_batch(plans, w_bits, grad_w_tilde, grad_w, grad_c, stream=None) -> None:
    """backward over lists; the gradient arrays are all float32 or all 16-bit
    (per list, chosen by element size as in backward)."""
    _same_len("backward_batch", plans, w_bits=w_bits, grad_w_tilde=grad_w_tilde, grad_w=grad_w, grad_c=grad_c)
    n = len(plans)
    flags = {_grad_flags(a, b) for a, b in zip(grad_w_tilde, grad_w)}
    if len(flags) != 1:
        raise ValueError("backward_batch: mixed 16-bit and float gradient arrays")
    f = flags.pop()
    pp, _a = _plans(plans)
    ns, ks = [p.n for p in plans], [p.k for p in plans]
    kk, _b = _parr(w_bits, 2, "w_bits", ns)
    g, _c = _parr(grad_w_tilde, 2 if f & GRAD_IN_HALF else 4, "grad_w_tilde", ns)
    gw, _d = _parr(grad_w, 2 if f & GRAD_OUT_HALF else 4, "grad_w", ns)
    gc, _e = _parr(grad_c, 4, "grad_c", ks)
    _check(_lib.edkm_backward_batch_ex(n, pp, kk, g, gw, gc, f, _stream(stream)), "backward_batch", plans)


def palettize_batch(plans, w_bits, lut, indices_out, stream=None) -> None:
    """palettize over a batch: one table launch and one packing launch per
    launch group (up to LAUNCH_GROUP matrices with the same bit width and format)."""
    _same_len("palettize_batch", plans, w_bits=w_bits, lut=lut, indices_out=indices_out)
    for p, o in zip(plans, indices_out):
        need = (p.n * p.bits + 7) // 8
        if o.numel() * o.element_size() < need:
            raise EdkmError(ERR_ARG, "palettize_batch", "indices_out needs %d bytes" % need)
    n = len(plans)
    pp, _a = _plans(plans)
    kk, _b = _parr(w_bits, 2, "w_bits", [p.n for p in plans])
    lt, _c = _parr(lut, 4, "lut", [p.k for p in plans])
    oo, _d = _parr(indices_out, 1, "indices_out", [(p.n * p.bits + 7) // 8 for p in plans])
    _check(_lib.edkm_palettize_batch(n, pp, kk, lt, oo, _stream(stream)), "palettize_batch", plans)


def unique_inverse_batch(plans, w_bits, unique_out=None, inverse_out=None, stream=None) -> None:
    """unique_inverse over a batch (list entries may be None where that output
    is not wanted): one ranking launch per launch group, plus one N-sized
    launch if any matrix of the group wants its inverse index."""
    _same_len("unique_inverse_batch", plans, w_bits=w_bits, unique_out=unique_out, inverse_out=inverse_out)
    n = len(plans)
    pp, _a = _plans(plans)
    ns = [p.n for p in plans]
    kk, _b = _parr(w_bits, 2, "w_bits", ns)
    uo, _c = _parr(unique_out, 2, "unique_out", [NKEYS] * n) if unique_out is not None else (None, None)
    io, _d = _parr(inverse_out, 2, "inverse_out", ns) if inverse_out is not None else (None, None)
    _check(_lib.edkm_unique_inverse_batch(n, pp, kk, uo, io, _stream(stream)), "unique_inverse_batch", plans)
