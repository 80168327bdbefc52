"""C-ABI checks that need no GPU: the library loads, exports every entry point
declared in include/edkm.h, sizes its workspace, and rejects bad arguments and
out-of-order calls on the host before any HIP call."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "edkm.h")

edkm = pytest.importorskip("paper_2309_00964_amd.edkm",
                           reason="libedkm.so not built (run __graft_entry__.build())")
lib = edkm._lib

FAKE_WS = 1 << 40          # a 256-byte-aligned address; plan_init never dereferences it


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(edkm_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) >= 11
    for name in names:
        assert hasattr(lib, name), name
    assert set(names) == set(edkm.EXPORTS)


def test_workspace_bytes():
    b = edkm.workspace_bytes(1 << 24, 3, 5)
    assert b > 0 and b % 256 == 0
    assert b < 64 << 20                      # independent of N, tens of MiB
    assert edkm.workspace_bytes(1, 3, 5) == b
    assert edkm.workspace_bytes(1 << 32 - 1, 3, 5) == b
    assert edkm.workspace_bytes(6_476_005_376, 3, 5) == 0   # above the per-matrix limit
    assert edkm.workspace_bytes(0, 3, 5) == 0
    assert edkm.workspace_bytes(10, 0, 5) == 0
    assert edkm.workspace_bytes(10, 5, 5) == 0
    assert edkm.workspace_bytes(10, 3, 0) == 0
    assert edkm.workspace_bytes(10, 3, 1025) == 0
    assert edkm.workspace_bytes(10, 3, 100) > b


def _plan(n=1000, bits=3, iters=5):
    p = edkm.edkm_plan()
    ws = edkm.workspace_bytes(n, bits, iters)
    assert lib.edkm_plan_init(ctypes.byref(p), n, bits, iters, FAKE_WS, ws) == edkm.OK
    return p


def test_plan_init_validation():
    p = edkm.edkm_plan()
    ws = edkm.workspace_bytes(1000, 3, 5)
    assert lib.edkm_plan_init(None, 1000, 3, 5, FAKE_WS, ws) == edkm.ERR_ARG
    assert lib.edkm_plan_init(ctypes.byref(p), 0, 3, 5, FAKE_WS, ws) == edkm.ERR_ARG
    assert lib.edkm_plan_init(ctypes.byref(p), 1000, 7, 5, FAKE_WS, ws) == edkm.ERR_ARG
    assert lib.edkm_plan_init(ctypes.byref(p), 1000, 3, 0, FAKE_WS, ws) == edkm.ERR_ARG
    assert lib.edkm_plan_init(ctypes.byref(p), 1000, 3, 5, None, ws) == edkm.ERR_WORKSPACE
    assert lib.edkm_plan_init(ctypes.byref(p), 1000, 3, 5, FAKE_WS, ws - 1) == edkm.ERR_WORKSPACE
    assert lib.edkm_plan_init(ctypes.byref(p), 1000, 3, 5, FAKE_WS + 16, ws) == edkm.ERR_WORKSPACE
    assert lib.edkm_plan_init(ctypes.byref(p), 1000, 3, 5, FAKE_WS, ws) == edkm.OK


def test_calls_out_of_order_are_rejected_before_any_gpu_work():
    p = _plan()
    keys = 1 << 41      # never dereferenced: rejected on the host first
    f = 1 << 42
    # forward and backward before init_unique
    assert lib.edkm_forward(ctypes.byref(p), keys, 2e-3, 0.0, f, f, f, 0, None, None) == edkm.ERR_STATE
    assert lib.edkm_backward(ctypes.byref(p), keys, f, f, f, None) == edkm.ERR_STATE
    assert lib.edkm_backward_dense(ctypes.byref(p), keys, f, f, f, None) == edkm.ERR_STATE
    assert lib.edkm_backward_ex(ctypes.byref(p), keys, f, f, f, 3, None) == edkm.ERR_STATE
    assert lib.edkm_backward_ex(ctypes.byref(p), keys, f, f, f, 4, None) == edkm.ERR_ARG   # unknown flag
    # an uninitialised plan is an argument error
    q = edkm.edkm_plan()
    assert lib.edkm_init_unique(ctypes.byref(q), keys, None, None, 0, None) == edkm.ERR_ARG
    assert lib.edkm_forward_dense(ctypes.byref(q), keys, 2e-3, 0.0, f, f, f, 0, None, None, None) == edkm.ERR_ARG


@pytest.mark.parametrize("tau,eps,fp16", [(0.0, 0.0, 0), (-1e-3, 0.0, 0), (float("inf"), 0.0, 0),
                                          (float("nan"), 0.0, 0), (1e-45, 0.0, 0), (2e-3, -1.0, 0),
                                          (2e-3, float("nan"), 0), (2e-3, 0.0, 2)])
def test_forward_argument_errors(tau, eps, fp16):
    p = _plan()
    keys, f = 1 << 41, 1 << 42
    assert lib.edkm_forward(ctypes.byref(p), keys, tau, eps, f, f, f, fp16, None, None) == edkm.ERR_ARG
    assert lib.edkm_forward_dense(ctypes.byref(p), keys, tau, eps, f, f, f, fp16, None, None, None) == edkm.ERR_ARG


def test_null_pointers_are_argument_errors():
    p = _plan()
    keys, f = 1 << 41, 1 << 42
    assert lib.edkm_init_unique(ctypes.byref(p), None, None, None, 0, None) == edkm.ERR_ARG
    assert lib.edkm_init_unique(ctypes.byref(p), keys, None, None, 2, None) == edkm.ERR_ARG
    assert lib.edkm_forward_dense(ctypes.byref(p), None, 2e-3, 0.0, f, f, f, 0, None, None, None) == edkm.ERR_ARG
    assert lib.edkm_forward_dense(ctypes.byref(p), keys, 2e-3, 0.0, None, f, f, 0, None, None, None) == edkm.ERR_ARG
    assert lib.edkm_forward_dense(ctypes.byref(p), keys, 2e-3, 0.0, f, None, f, 0, None, None, None) == edkm.ERR_ARG
    assert lib.edkm_forward_dense(ctypes.byref(p), keys, 2e-3, 0.0, f, f, None, 0, None, None, None) == edkm.ERR_ARG
    assert lib.edkm_backward_dense(ctypes.byref(p), keys, None, f, f, None) == edkm.ERR_ARG


def test_unique_inverse_argument_and_state_errors():
    p = _plan()
    keys, u = 1 << 41, 1 << 42
    # no output at all
    assert lib.edkm_unique_inverse(ctypes.byref(p), keys, None, None, None) == edkm.ERR_ARG
    assert lib.edkm_unique_inverse(ctypes.byref(p), None, u, None, None) == edkm.ERR_ARG
    # before init_unique: nothing to rank
    assert lib.edkm_unique_inverse(ctypes.byref(p), keys, u, None, None) == edkm.ERR_STATE
    assert lib.edkm_unique_inverse(ctypes.byref(p), keys, None, u, None) == edkm.ERR_STATE
    q = edkm.edkm_plan()
    assert lib.edkm_unique_inverse(ctypes.byref(q), keys, u, u, None) == edkm.ERR_ARG
    # batch: one matrix without either output is an argument error
    p2 = edkm.edkm_plan()
    ws = edkm.workspace_bytes(1000, 3, 5)
    assert lib.edkm_plan_init(ctypes.byref(p2), 1000, 3, 5, FAKE_WS + ws + (256 - ws % 256) % 256, ws) == edkm.OK
    arr = (ctypes.c_void_p * 2)(ctypes.addressof(p), ctypes.addressof(p2))
    kk = (ctypes.c_void_p * 2)(keys, keys)
    uo = (ctypes.c_void_p * 2)(u, None)
    pp, kp, up = (ctypes.cast(x, edkm._PP) for x in (arr, kk, uo))
    assert lib.edkm_unique_inverse_batch(2, pp, kp, up, None, None) == edkm.ERR_ARG
    uo[1] = u
    assert lib.edkm_unique_inverse_batch(2, pp, kp, up, None, None) == edkm.ERR_STATE


def test_batch_argument_errors():
    p1, p2 = _plan(), _plan()
    arr = (ctypes.c_void_p * 2)(ctypes.addressof(p1), ctypes.addressof(p1))
    keys = (ctypes.c_void_p * 2)(1 << 41, 1 << 41)
    pp = ctypes.cast(arr, edkm._PP)
    kk = ctypes.cast(keys, edkm._PP)
    # the same plan twice, or plans sharing a workspace
    assert lib.edkm_init_unique_batch(2, pp, kk, None, None, 0, None) == edkm.ERR_ARG
    arr[1] = ctypes.addressof(p2)
    assert lib.edkm_init_unique_batch(2, pp, kk, None, None, 0, None) == edkm.ERR_ARG
    assert lib.edkm_init_unique_batch(0, pp, kk, None, None, 0, None) == edkm.ERR_ARG
    assert lib.edkm_init_unique_batch(2, None, kk, None, None, 0, None) == edkm.ERR_ARG


def test_palettize_batch_argument_errors():
    p, q = _plan(), _plan()          # q shares p's (fake) workspace
    one = lambda v: ctypes.cast((ctypes.c_void_p * 1)(v), edkm._PP)
    pp, kk, good, nul = one(ctypes.addressof(p)), one(1 << 41), one(1 << 42), one(None)
    assert lib.edkm_palettize_batch(1, pp, kk, None, good, None) == edkm.ERR_ARG
    assert lib.edkm_palettize_batch(1, pp, kk, good, None, None) == edkm.ERR_ARG
    assert lib.edkm_palettize_batch(1, pp, kk, nul, good, None) == edkm.ERR_ARG
    assert lib.edkm_palettize_batch(1, pp, kk, good, nul, None) == edkm.ERR_ARG
    assert lib.edkm_palettize_batch(1, pp, nul, good, good, None) == edkm.ERR_ARG
    assert lib.edkm_palettize_batch(0, pp, kk, good, good, None) == edkm.ERR_ARG
    assert lib.edkm_palettize_batch(1, None, kk, good, good, None) == edkm.ERR_ARG
    two = ctypes.cast((ctypes.c_void_p * 2)(ctypes.addressof(p), ctypes.addressof(q)), edkm._PP)
    k2 = ctypes.cast((ctypes.c_void_p * 2)(1 << 41, 1 << 41), edkm._PP)
    g2 = ctypes.cast((ctypes.c_void_p * 2)(1 << 42, 1 << 42), edkm._PP)
    assert lib.edkm_palettize_batch(2, two, k2, g2, g2, None) == edkm.ERR_ARG


def test_batch_bindings_reject_lists_of_other_lengths():
    """The C side reads `count` entries of every host array: a short list must
    be refused by the binding before the library is called."""
    from types import SimpleNamespace
    plans = [SimpleNamespace(n=100, bits=3), SimpleNamespace(n=100, bits=3)]
    one, two = [object()], [object(), object()]
    with pytest.raises(edkm.EdkmError, match="w_bits has 1 entries"):
        edkm.init_unique_batch(plans, one)
    with pytest.raises(edkm.EdkmError, match="num_unique_out"):
        edkm.init_unique_batch(plans, two, num_unique_out=one)
    with pytest.raises(edkm.EdkmError, match="c_out"):
        edkm.forward_batch(plans, two, 2e-3, 0.0, two, one, two)
    with pytest.raises(edkm.EdkmError, match="iters_out"):
        edkm.forward_batch(plans, two, 2e-3, 0.0, two, two, two, iters_out=one)
    with pytest.raises(edkm.EdkmError, match="grad_c"):
        edkm.backward_batch(plans, two, two, two, one)
    with pytest.raises(edkm.EdkmError, match="lut"):
        edkm.palettize_batch(plans, two, one, two)
    with pytest.raises(edkm.EdkmError, match="indices_out"):
        edkm.palettize_batch(plans, two, two, [object(), object(), object()])


def test_launch_group_size_matches_header():
    text = open(HEADER).read()
    assert int(re.search(r"#define EDKM_LAUNCH_GROUP (\d+)", text).group(1)) == edkm.LAUNCH_GROUP


class _FakeDeviceTensor:
    """Just enough of a tensor for the binding's checks (no GPU here).  Its
    address is never dereferenced: an undersized one must be refused while the
    arguments are marshalled, and should a check be missing, the stub plan (a
    NULL record) makes the library reject the call on the host, which the
    test's match on the argument name reports."""

    def __init__(self, numel, esize):
        self._n, self._e = numel, esize
        self.is_cuda = True

    def is_contiguous(self):
        return True

    def element_size(self):
        return self._e

    def numel(self):
        return self._n

    def data_ptr(self):
        return 1 << 40


def test_binding_refuses_undersized_tensors():
    from types import SimpleNamespace
    plan = SimpleNamespace(n=1000, bits=3, k=8, ref=None, plan=edkm.edkm_plan())   # a zeroed record: rejected on the host
    f = _FakeDeviceTensor
    keys, short_keys = f(1000, 2), f(999, 2)
    c, short_c = f(8, 4), f(7, 4)
    vec, short_vec = f(1000, 4), f(999, 4)
    cases = [
        (lambda: edkm.init_unique(plan, short_keys), "w_bits"),
        (lambda: edkm.init_unique(plan, keys, counts_out=f(65535, 4)), "counts_out"),
        (lambda: edkm.forward(plan, keys, 2e-3, 0.0, short_c, c, vec), "c_in"),
        (lambda: edkm.forward(plan, keys, 2e-3, 0.0, c, short_c, vec), "c_out"),
        (lambda: edkm.forward(plan, keys, 2e-3, 0.0, c, c, short_vec), "w_tilde"),
        (lambda: edkm.forward(plan, keys, 2e-3, 0.0, c, c, f(999, 2), out_half=True), "w_tilde"),
        (lambda: edkm.backward(plan, keys, short_vec, vec, c), "grad_w_tilde"),
        (lambda: edkm.backward(plan, keys, vec, short_vec, c), "grad_w"),
        (lambda: edkm.backward(plan, keys, vec, vec, short_c), "grad_c"),
        (lambda: edkm.forward_dense(plan, keys, 2e-3, 0.0, c, c, vec, attn_out=f(7999, 4)), "attn_out"),
        (lambda: edkm.backward_dense(plan, short_keys, vec, vec, c), "w_bits"),
        (lambda: edkm.palettize(plan, keys, short_c, f(375, 1)), "lut"),
        (lambda: edkm.forward_batch([plan, plan], [keys, keys], 2e-3, 0.0, [c, c], [c, c], [vec, short_vec]),
         r"w_tilde\[1\]"),
        (lambda: edkm.backward_batch([plan], [keys], [vec], [vec], [short_c]), r"grad_c\[0\]"),
        (lambda: edkm.palettize_batch([plan], [keys], [c], [f(374, 1)]), "indices_out"),
    ]
    for call, what in cases:
        with pytest.raises((ValueError, edkm.EdkmError), match=what):
            call()


def test_status_strings():
    for s in (0, -1, -2, -3, -4, -5):
        assert edkm.status_str(s) and edkm.status_str(s) != "unknown status"
    assert edkm.status_str(-99) == "unknown status"


def test_pass_event_ids_match_header():
    text = open(HEADER).read()
    ids = dict((k, int(v)) for k, v in re.findall(r"\bEDKM_(PASS_[A-Z_]+)\s*=\s*(\d+)", text))
    assert ids == {name: getattr(edkm, name) for name in ids}
    assert sorted(ids.values()) == list(range(len(ids)))
    p = _plan()
    for pid in ids.values():     # NULL events switch the hook off: host only
        assert lib.edkm_plan_set_pass_events(ctypes.byref(p), pid, None, None) == edkm.OK
    assert lib.edkm_plan_set_pass_events(ctypes.byref(p), len(ids), None, None) == edkm.ERR_ARG
    assert lib.edkm_plan_set_pass_events(ctypes.byref(p), -1, None, None) == edkm.ERR_ARG


def test_keyed_mode_setting():
    p = _plan()
    for mode in (edkm.KEYED_AUTO, edkm.KEYED_I32, edkm.KEYED_U64):
        assert lib.edkm_plan_set_keyed_mode(ctypes.byref(p), mode) == edkm.OK
    assert lib.edkm_plan_set_keyed_mode(ctypes.byref(p), -2) == edkm.ERR_ARG
    assert lib.edkm_plan_set_keyed_mode(ctypes.byref(p), 2) == edkm.ERR_ARG
    assert lib.edkm_plan_set_keyed_mode(None, 0) == edkm.ERR_ARG


def test_plan_init_ex_key_formats():
    p = edkm.edkm_plan()
    ws = edkm.workspace_bytes(1000, 3, 5)
    for fmt in (edkm.KEYS_FP16, edkm.KEYS_BF16):
        assert lib.edkm_plan_init_ex(ctypes.byref(p), 1000, 3, 5, fmt, FAKE_WS, ws) == edkm.OK
    for fmt in (-1, 2):
        assert lib.edkm_plan_init_ex(ctypes.byref(p), 1000, 3, 5, fmt, FAKE_WS, ws) == edkm.ERR_ARG


def test_plan_record_size_matches_header():
    m = re.search(r"uint64_t\s+opaque\[(\d+)\]", open(HEADER).read())
    assert m and ctypes.sizeof(edkm.edkm_plan) == 8 * int(m.group(1))


def test_plain_c_consumer_compiles_and_gets_host_errors(tmp_path):
    """tests/abi_consumer.c, a plain C program, compiles with gcc against
    include/edkm.h alone (no platform define on the command line), links the
    built library and sees the documented host-side errors, a copied plan
    record included."""
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not available")
    libdir = os.path.dirname(os.path.abspath(edkm._lib._name))
    exe = str(tmp_path / "abi_consumer")
    subprocess.check_call([gcc, "-std=c99", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"),
                           "-I", "/opt/rocm/include", os.path.join(ROOT, "tests", "abi_consumer.c"),
                           "-L", libdir, "-ledkm", "-Wl,-rpath," + libdir, "-o", exe])
    out = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert out.returncode == 0, out.stdout + out.stderr
    assert out.stdout.strip() == "ok"


def test_palettize_noalloc_argument_errors():
    """The allocation-free palettization rejects bad arguments on the host,
    before its device-address lookup or any launch."""
    keys, lut, out = 1 << 41, 1 << 42, 1 << 43   # never dereferenced
    f = lib.edkm_palettize_noalloc
    assert f(None, 100, 3, edkm.KEYS_FP16, lut, out, None) == edkm.ERR_ARG
    assert f(keys, 100, 3, edkm.KEYS_FP16, None, out, None) == edkm.ERR_ARG
    assert f(keys, 100, 3, edkm.KEYS_FP16, lut, None, None) == edkm.ERR_ARG
    assert f(keys, 0, 3, edkm.KEYS_FP16, lut, out, None) == edkm.ERR_ARG
    assert f(keys, (1 << 32), 3, edkm.KEYS_FP16, lut, out, None) == edkm.ERR_ARG   # above EDKM_MAX_N
    assert f(keys, 100, 0, edkm.KEYS_FP16, lut, out, None) == edkm.ERR_ARG
    assert f(keys, 100, 5, edkm.KEYS_FP16, lut, out, None) == edkm.ERR_ARG
    assert f(keys, 100, 3, 2, lut, out, None) == edkm.ERR_ARG
    text = open(HEADER).read()
    assert re.search(r"#define EDKM_NOALLOC_SCRATCH_BYTES 65536\b", text)


def test_differentiable_wrapper_argument_errors():
    """function.dkm checks its arguments on the host before any HIP call."""
    import torch
    from paper_2309_00964_amd.function import dkm
    c8 = torch.zeros(8)
    with pytest.raises(TypeError):
        dkm(torch.zeros(16, dtype=torch.float16), c8)           # not on the GPU
    with pytest.raises(TypeError):
        dkm(torch.zeros(16, dtype=torch.float32), c8)           # not 16-bit weights


def test_backward_gradient_flags_follow_element_sizes():
    """The binding picks edkm_backward_ex's flags from the gradient arrays:
    2-byte elements are 16-bit floats of the plan's format, 4-byte ones float."""
    import torch
    f32, h = torch.zeros(4), torch.zeros(4, dtype=torch.int16)
    assert edkm._grad_flags(f32, f32) == 0
    assert edkm._grad_flags(h, f32) == edkm.GRAD_IN_HALF
    assert edkm._grad_flags(f32, h) == edkm.GRAD_OUT_HALF
    assert edkm._grad_flags(h, h) == edkm.GRAD_IN_HALF | edkm.GRAD_OUT_HALF
    with pytest.raises(ValueError):
        edkm._grad_flags(torch.zeros(4, dtype=torch.float64), f32)
