"""CPU emulation of generic-kernel plans against the oracle (no GPU).

The host planner is compiled together with a CPU executor of the generic
kernel's descriptor semantics (tests/cpu_emulator/emulate.cpp, with UBSan);
every launch's reads and writes are bounds-checked.  Forward and backward of
every workload at reduced size must match the float64 oracle."""
import ctypes as C
import os
import subprocess

import numpy as np
import pytest

import oracle as O
import workloads as W
from conftest import CIRCULAR_CASES, EDGE_CASES, STRIDED_CASES, strides_of, PAPER_SHAPES, ROOT, load_layer_strings

STRINGS = load_layer_strings()

SRC = os.path.join(ROOT, "paper_2401_03384_amd", "csrc")


@pytest.fixture(scope="module")
def emul(tmp_path_factory):
    out = str(tmp_path_factory.mktemp("emul") / "libce_emul.so")
    cmd = ["g++", "-O1", "-g", "-shared", "-fPIC", "-std=c++17", "-fsanitize=undefined",
           "-fno-sanitize-recover=undefined", "-I", os.path.join(ROOT, "include"), "-I", SRC,
           os.path.join(ROOT, "tests", "cpu_emulator", "emulate.cpp"),
           os.path.join(SRC, "expr.cpp"), os.path.join(SRC, "plan.cpp"),
           os.path.join(SRC, "lower.cpp"), os.path.join(SRC, "fuse.cpp"), os.path.join(SRC, "fuse_rcp.cpp"),
           os.path.join(SRC, "fuse_tt.cpp"),
           os.path.join(SRC, "capi.cpp"), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        pytest.fail(r.stderr)
    L = C.CDLL(out)
    L.emul_run.restype = C.c_int
    return L


def _to_storage(a, bf16):
    a32 = np.ascontiguousarray(a, dtype=np.float32)
    return W.bf16_bits(a32) if bf16 else a32


def _from_storage(a, bf16):
    if bf16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def _run(L, spec, shapes, bf16, mode, ins, dy=None, out_shape=None, feature=0, generic=1):
    n = len(shapes)
    ranks = (C.c_int * n)(*[len(s) for s in shapes])
    bufs = [(C.c_int64 * len(s))(*s) for s in shapes]
    dims = (C.POINTER(C.c_int64) * n)(*[C.cast(b, C.POINTER(C.c_int64)) for b in bufs])
    st = [_to_storage(a, bf16) for a in ins]
    inp = (C.c_void_p * n)(*[a.ctypes.data for a in st])
    err = C.create_string_buffer(512)
    if mode == 0:
        out = np.zeros(out_shape, dtype=np.uint16 if bf16 else np.float32)
        rc = L.emul_run(spec.encode(), n, ranks, dims, int(bf16), 0, inp, out.ctypes.data_as(C.c_void_p),
                        None, None, err, 512, generic)
        assert rc == 0, err.value.decode()
        return _from_storage(out, bf16)
    d = _to_storage(dy, bf16)
    grads = [np.zeros(s, dtype=(np.uint16 if (bf16 and i == feature) else np.float32))
             for i, s in enumerate(shapes)]
    din = (C.c_void_p * n)(*[g.ctypes.data for g in grads])
    rc = L.emul_run(spec.encode(), n, ranks, dims, int(bf16), 1, inp, None,
                    d.ctypes.data_as(C.c_void_p), din, err, 512, generic)
    assert rc == 0, err.value.decode()
    return [_from_storage(g, bf16 and i == feature) for i, g in enumerate(grads)]


def _rel(a, b):
    return float(np.linalg.norm((a - b).ravel()) / max(np.linalg.norm(b.ravel()), 1e-300))


# the parity strings at sizes a CPU emulation finishes quickly (ragged spatial sizes)
CASES = {
    "C1": W.PARITY_WORKLOADS["C1"],
    "C2s": W.PARITY_WORKLOADS["C2s"],
    "C2s_bf16": W.PARITY_WORKLOADS["C2s_bf16"],
    "C2r32": W.cp_layer("C2r32t", 2, 32, 32, 5, 37, 32, 3, "f32", 17),
    "C2r32_bf16": W.cp_layer("C2r32t_bf16", 2, 32, 32, 5, 37, 32, 3, "bf16", 17),
    "C2k5": W.cp_layer("C2k5t", 1, 32, 32, 6, 29, 32, 5, "f32", 18),
    # fused CP chains with ranks below 32
    "C2r16": W.cp_layer("C2r16t", 2, 32, 32, 5, 37, 16, 3, "f32", 26),
    "C2r8_bf16": W.cp_layer("C2r8t_bf16", 2, 32, 64, 5, 19, 8, 3, "bf16", 27),
    "C2r20k5": W.cp_layer("C2r20k5t", 1, 32, 32, 6, 29, 20, 5, "f32", 28),
    # channel counts off the 32 / 64 blocks
    "C2c48": W.cp_layer("C2c48t", 2, 48, 40, 5, 37, 24, 3, "f32", 29),
    "C2c16_bf16": W.cp_layer("C2c16t_bf16", 2, 16, 16, 5, 19, 8, 3, "bf16", 30),
    "C2c20k5": W.cp_layer("C2c20k5t", 1, 20, 56, 6, 29, 32, 5, "f32", 31),
    "C3t": W.tucker2_layer("C3t", 2, 32, 24, 7, 9, 8, 16, 3, "bf16", 21),
    "C3t_f32": W.tucker2_layer("C3t_f32", 2, 32, 24, 7, 9, 8, 16, 3, "f32", 21),
    # Tucker cores on MFMA tiles (ragged channels, 5 x 5 taps, row tiles)
    "C3c": W.PARITY_WORKLOADS["C3c"],
    "C3c5": W.PARITY_WORKLOADS["C3c5"],
    "C3m": W.PARITY_WORKLOADS["C3m"],
    "C3c_f32": W.PARITY_WORKLOADS["C3c_f32"],
    "C3p5": W.PARITY_WORKLOADS["C3p5"],
    "C4c": W.PARITY_WORKLOADS["C4c"],
    "C4t": W.rtt_layer("C4t", 1, (2, 4, 2), (2, 2, 4), 7, 6, 4, 3, "f32", 22),
    "C5at": W.rcp_layer("C5at", 2, (4, 2, 4), (2, 4, 2), 5, 7, 16, 3, "bf16", 23),
    "C5at_f32": W.rcp_layer("C5at_f32", 2, (4, 2, 4), (2, 4, 2), 5, 7, 16, 3, "f32", 23),
    "C5bt": W.rcp_layer("C5bt", 1, (2, 2, 4), (2, 2, 4), 9, 8, 16, 5, "bf16", 24),
    "C4m": W.rtt_layer("C4m", 1, (4, 4, 8), (4, 4, 8), 5, 7, 16, 3, "f32", 26),
    # fused contraction + convolution: 30, 40 and 16 columns, ragged bands, t3 < 8, K1 = 24
    "C4x2": W.PARITY_WORKLOADS["C4x2"],
    "C4x4": W.PARITY_WORKLOADS["C4x4"],
    "C4x1": W.PARITY_WORKLOADS["C4x1"],
    # transposed convolution with register-held filter operands: a partial q
    # tile with 7 channels, a 2 x 2 filter, two row tiles
    "C4q": W.PARITY_WORKLOADS["C4q"],
    "C4k2": W.PARITY_WORKLOADS["C4k2"],
    "C4p": W.PARITY_WORKLOADS["C4p"],
    "C5cs": W.PARITY_WORKLOADS["C5cs"],
    # fused reshaped-CP kernels: both instantiations (rank 4 keeps the CPU
    # run short), one and several row tiles
    "C5ar": W.rcp_layer("C5ar", 2, (8, 8, 8), (8, 8, 8), 7, 7, 4, 3, "bf16", 29),
    "C5br": W.rcp_layer("C5br", 1, (4, 4, 8), (4, 4, 8), 11, 11, 4, 5, "bf16", 30),
    "C5bt2": W.PARITY_WORKLOADS["C5bt2"],
    "C5bt3": W.PARITY_WORKLOADS["C5bt3"],
    "C5cs_f32": W.PARITY_WORKLOADS["C5cs_f32"],
}


@pytest.mark.parametrize("generic", [1, 0], ids=["generic", "fast"])
@pytest.mark.parametrize("name", sorted(CASES))
def test_emulated_plan_matches_oracle(emul, name, generic):
    w = CASES[name]
    bf16 = w.dtype == "bf16"
    tol = 2e-2 if bf16 else 1e-5
    ins, dy = W.make_inputs(w)
    e = O.bind(O.parse(w.spec), w.shapes)
    tree = O.optimal_tree(e)[0]
    y_ref = O.eval_pairwise(e, ins, tree)
    y = _run(emul, w.spec, w.shapes, bf16, 0, ins, out_shape=w.out_shape, generic=generic)
    assert _rel(y, y_ref) <= tol
    if not w.backward:
        return
    g_ref = O.grads_pairwise(e, ins, tree, dy)
    g = _run(emul, w.spec, w.shapes, bf16, 1, ins, dy=dy, generic=generic)
    for i, (a, b) in enumerate(zip(g, g_ref)):
        assert _rel(a, b) <= tol, (name, i, _rel(a, b))


@pytest.mark.parametrize("generic", [1, 0], ids=["generic", "fast"])
@pytest.mark.parametrize("spec,shapes", [
    ("bsh,tsh->bth|h", [(2, 3, 11), (4, 3, 4)]),                 # even filter
    ("tsh,bsh->bth|h", [(4, 3, 3), (2, 3, 9)]),                  # feature second
    ("bshw,sh,sw->bshw|hw", [(2, 3, 7, 6), (3, 3), (3, 5)]),     # depthwise
    ("bsm,mt->bt", [(2, 3, 4), (4, 5)]),                          # self-contraction
    ("ij->ji", [(3, 4)]),                                         # single operand
    ("ijk->i", [(3, 4, 2)]),                                      # single operand, sums
    ("bshw,(r1)t,(r1)(r2)h,(r2)(r3)w,(r3)s->bthw|hw",
     [(2, 3, 6, 5), (2, 4), (2, 3, 3), (3, 2, 3), (2, 3)]),       # tensor-train
    ("bshw,(r0)(r1)t,(r1)(r2)h,(r2)(r3)w,(r3)(r0)s->bthw|hw",
     [(1, 3, 6, 5), (2, 2, 4), (2, 2, 3), (2, 2, 3), (2, 2, 3)]),  # tensor-ring
])
def test_emulated_plan_edge_cases(emul, spec, shapes, generic):
    e = O.bind(O.parse(spec), shapes)
    g0 = np.random.default_rng(3)
    ins = [g0.standard_normal(s).astype(np.float32).astype(np.float64) for s in shapes]
    out_shape = tuple(e.out_sizes[l] for l in e.output)
    dy = g0.standard_normal(out_shape).astype(np.float32).astype(np.float64)
    tree = O.optimal_tree(e)[0] if e.n > 1 else 0
    y_ref = O.eval_pairwise(e, ins, tree)
    y = _run(emul, spec, shapes, False, 0, ins, out_shape=out_shape, generic=generic)
    assert _rel(y, y_ref) <= 1e-6
    if e.n > 1:
        g_ref = O.grads_pairwise(e, ins, tree, dy)
    else:
        g_ref = [np.broadcast_to(np.einsum(
            "".join(chr(97 + k) for k in range(len(e.output))) + "->" +
            "".join(chr(97 + e.output.index(l)) if l in e.output else "" for l in e.inputs[0]),
            dy).reshape([s if l in e.output else 1 for l, s in zip(e.inputs[0], shapes[0])]),
            shapes[0])]
    g = _run(emul, spec, shapes, False, 1, ins, dy=dy, generic=generic)
    for a, b in zip(g, g_ref):
        assert _rel(a, b) <= 1e-6


def _run_saved(L, spec, shapes, bf16, ins, dy, out_shape, flags):
    """Forward then backward on one workspace (mode 2)."""
    n = len(shapes)
    ranks = (C.c_int * n)(*[len(s) for s in shapes])
    bufs = [(C.c_int64 * len(s))(*s) for s in shapes]
    dims = (C.POINTER(C.c_int64) * n)(*[C.cast(b, C.POINTER(C.c_int64)) for b in bufs])
    st = [_to_storage(a, bf16) for a in ins]
    inp = (C.c_void_p * n)(*[a.ctypes.data for a in st])
    err = C.create_string_buffer(512)
    out = np.zeros(out_shape, dtype=np.uint16 if bf16 else np.float32)
    d = _to_storage(dy, bf16)
    grads = [np.zeros(s, dtype=(np.uint16 if (bf16 and i == 0) else np.float32)) for i, s in enumerate(shapes)]
    din = (C.c_void_p * n)(*[g.ctypes.data for g in grads])
    rc = L.emul_run(spec.encode(), n, ranks, dims, int(bf16), 2, inp, out.ctypes.data_as(C.c_void_p),
                    d.ctypes.data_as(C.c_void_p), din, err, 512, flags)
    assert rc == 0, err.value.decode()
    return _from_storage(out, bf16), [_from_storage(g, bf16 and i == 0) for i, g in enumerate(grads)]


SAVE = 0x4   # CE_FLAG_SAVE_INTERMEDIATES


@pytest.mark.parametrize("flags", [SAVE, SAVE | 0x1], ids=["fast", "generic"])
@pytest.mark.parametrize("name", ["C2s", "C3t", "C4t", "C5at_f32", "C5br"])
def test_saved_intermediates(emul, name, flags):
    """With the forward's intermediates kept in the workspace the backward
    skips the recompute launches and still matches the oracle."""
    w = CASES[name]
    bf16 = w.dtype == "bf16"
    tol = 2e-2 if bf16 else 1e-5
    ins, dy = W.make_inputs(w)
    e = O.bind(O.parse(w.spec), w.shapes)
    tree = O.optimal_tree(e)[0]
    y, g = _run_saved(emul, w.spec, w.shapes, bf16, ins, dy, w.out_shape, flags)
    assert _rel(y, O.eval_pairwise(e, ins, tree)) <= tol
    for a, b in zip(g, O.grads_pairwise(e, ins, tree, dy)):
        assert _rel(a, b) <= tol


@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
@pytest.mark.parametrize("name", sorted(PAPER_SHAPES))
def test_emulated_paper_strings(emul, name, bf16):
    """Every executable layer string the paper prints, default plan (the same
    launches the GPU runs), forward and backward, bounds-checked, vs the oracle."""
    spec = STRINGS[name][0]
    shapes = PAPER_SHAPES[name]
    e = O.bind(O.parse(spec), shapes)
    tol = 2e-2 if bf16 else 1e-5
    rng = np.random.default_rng(7)
    ins = [rng.standard_normal(s).astype(np.float32) for s in shapes]
    ins = [(W.round_to_bf16(a) if bf16 else a).astype(np.float64) for a in ins]
    out_shape = tuple(e.out_sizes[l] for l in e.output)
    dy = rng.standard_normal(out_shape).astype(np.float32)
    dy = (W.round_to_bf16(dy) if bf16 else dy).astype(np.float64)
    tree = O.optimal_tree(e)[0]
    y = _run(emul, spec, shapes, bf16, 0, ins, out_shape=out_shape, generic=0)
    assert _rel(y, O.eval_pairwise(e, ins, tree)) <= tol
    g = _run(emul, spec, shapes, bf16, 1, ins, dy=dy, generic=0)
    for a, b in zip(g, O.grads_pairwise(e, ins, tree, dy)):
        assert _rel(a, b) <= tol


@pytest.mark.parametrize("name", ["C4t", "C5at"])
def test_emulated_memory_limited(emul, name):
    """The memory-limited order (cap just below the optimum's largest
    intermediate), every launch bounds-checked, against the oracle along the
    oracle's limited tree."""
    w = CASES[name]
    bf16 = w.dtype == "bf16"
    tol = 2e-2 if bf16 else 1e-5
    ins, dy = W.make_inputs(w)
    e = O.bind(O.parse(w.spec), w.shapes)
    cap = O.max_intermediate(e, O.optimal_tree(e)[0]) - 1
    tree, _ = O.optimal_tree(e, max_elements=cap)
    assert tree is not None
    emul.emul_set_limit(C.c_uint64(cap))
    try:
        y = _run(emul, w.spec, w.shapes, bf16, 0, ins, out_shape=w.out_shape, generic=0)
        g = _run(emul, w.spec, w.shapes, bf16, 1, ins, dy=dy, generic=0)
    finally:
        emul.emul_set_limit(C.c_uint64(0))
    assert _rel(y, O.eval_pairwise(e, ins, tree)) <= tol
    for a, b in zip(g, O.grads_pairwise(e, ins, tree, dy)):
        assert _rel(a, b) <= tol


@pytest.mark.parametrize("name,flags", [("C2s", 0x2), ("C3t", 0), ("C4t", 0), ("C5at_f32", 0),
                                        ("C5br", 0x2)])
def test_emulated_save_budget(emul, name, flags):
    """Checkpointing under a save budget (half the intermediates' bytes):
    the forward keeps the chosen intermediates, the backward reads them and
    recomputes the rest on one bounds-checked workspace; vs the oracle."""
    w = CASES[name]
    bf16 = w.dtype == "bf16"
    tol = 2e-2 if bf16 else 1e-5
    ins, dy = W.make_inputs(w)
    e = O.bind(O.parse(w.spec), w.shapes)
    tree = O.optimal_tree(e)[0]
    total = O.checkpoint_choice(e, tree, 10 ** 18, 2 if bf16 else 4)[1]
    emul.emul_set_save_budget(C.c_uint64(total // 2))
    try:
        y, g = _run_saved(emul, w.spec, w.shapes, bf16, ins, dy, w.out_shape, flags)
    finally:
        emul.emul_set_save_budget(C.c_uint64(0))
    assert _rel(y, O.eval_pairwise(e, ins, tree)) <= tol
    for a, b in zip(g, O.grads_pairwise(e, ins, tree, dy)):
        assert _rel(a, b) <= tol


@pytest.mark.parametrize("generic", [0, 1], ids=["fast", "generic"])
@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
@pytest.mark.parametrize("name", sorted(STRIDED_CASES))
def test_emulated_strided(emul, name, bf16, generic):
    """Strided convolutions (Appendix B varieties): forward, and the backward
    whose transposed convolutions run as stride-1 phases on views of the
    gradient and the filter; every access bounds-checked; vs the oracle."""
    spec, shapes, st = STRIDED_CASES[name]
    e = O.bind(O.parse(spec), shapes, strides=strides_of(st))
    tol = 2e-2 if bf16 else 1e-5
    rng = np.random.default_rng(9)
    ins = [rng.standard_normal(s).astype(np.float32) for s in shapes]
    ins = [(W.round_to_bf16(a) if bf16 else a).astype(np.float64) for a in ins]
    out_shape = tuple(e.out_sizes[l] for l in e.output)
    dy = rng.standard_normal(out_shape).astype(np.float32)
    dy = (W.round_to_bf16(dy) if bf16 else dy).astype(np.float64)
    tree = O.optimal_tree(e)[0]
    emul.emul_set_strides(st.encode())
    try:
        y = _run(emul, spec, shapes, bf16, 0, ins, out_shape=out_shape, generic=generic)
        g = _run(emul, spec, shapes, bf16, 1, ins, dy=dy, generic=generic)
    finally:
        emul.emul_set_strides(b"")
    assert _rel(y, O.eval_pairwise(e, ins, tree)) <= tol
    for a, b in zip(g, O.grads_pairwise(e, ins, tree, dy)):
        assert _rel(a, b) <= tol


@pytest.mark.parametrize("order", ["optimal", "ltr"])
@pytest.mark.parametrize("name", ["conv1", "conv3_1", "conv3_sc", "conv5_x"])
def test_emulated_resnet34_cp_layers(emul, name, order):
    """ResNet-34 convolutions as CP layers at reduced size, the planned and
    the left-to-right order, every launch bounds-checked, vs the oracle."""
    w, strides = W.resnet34_cp_layer(name, batch=1, scale=8)
    ins, dy = W.make_inputs(w)
    e = O.bind(O.parse(w.spec), w.shapes, strides=strides)
    tree = O.left_to_right_tree(5) if order == "ltr" else O.optimal_tree(e)[0]
    st = ",".join(f"{k}={v}" for k, v in strides.items())
    emul.emul_set_strides(st.encode())
    emul.emul_set_path(1 if order == "ltr" else 0)
    try:
        y = _run(emul, w.spec, w.shapes, False, 0, ins, out_shape=w.out_shape, generic=0)
        g = _run(emul, w.spec, w.shapes, False, 1, ins, dy=dy, generic=0)
    finally:
        emul.emul_set_strides(b"")
        emul.emul_set_path(0)
    assert _rel(y, O.eval_pairwise(e, ins, tree)) <= 1e-5
    for a, b in zip(g, O.grads_pairwise(e, ins, tree, dy)):
        assert _rel(a, b) <= 1e-5


@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
@pytest.mark.parametrize("name", sorted(CIRCULAR_CASES))
def test_emulated_circular(emul, name, bf16):
    """Circular convolutions (two-, three- and four-way), every access of the
    generic kernel's modulo positions bounds-checked, against the oracle."""
    spec, shapes, circ = CIRCULAR_CASES[name]
    e = O.bind(O.parse(spec), shapes, circular=circ)
    tol = 2e-2 if bf16 else 1e-5
    rng = np.random.default_rng(5)
    ins = [rng.standard_normal(s).astype(np.float32) for s in shapes]
    ins = [(W.round_to_bf16(a) if bf16 else a).astype(np.float64) for a in ins]
    out_shape = tuple(e.out_sizes[l] for l in e.output)
    dy = rng.standard_normal(out_shape).astype(np.float32)
    dy = (W.round_to_bf16(dy) if bf16 else dy).astype(np.float64)
    tree = O.optimal_tree(e)[0]
    emul.emul_set_circular(",".join(circ).encode())
    try:
        y = _run(emul, spec, shapes, bf16, 0, ins, out_shape=out_shape, generic=0)
        g = _run(emul, spec, shapes, bf16, 1, ins, dy=dy, generic=0)
    finally:
        emul.emul_set_circular(b"")
    assert _rel(y, O.eval_pairwise(e, ins, tree)) <= tol
    for a, b in zip(g, O.grads_pairwise(e, ins, tree, dy)):
        assert _rel(a, b) <= tol


@pytest.mark.parametrize("name", ["conv3d", "conv4d"])
def test_emulated_convnd(emul, name):
    """Three and four convolved labels in one step (Section 3.1: conv3d and
    beyond), bounds-checked, vs the oracle."""
    spec, shapes, _ = EDGE_CASES[name]
    e = O.bind(O.parse(spec), shapes)
    rng = np.random.default_rng(6)
    ins = [rng.standard_normal(s).astype(np.float32).astype(np.float64) for s in shapes]
    out_shape = tuple(e.out_sizes[l] for l in e.output)
    dy = rng.standard_normal(out_shape).astype(np.float32).astype(np.float64)
    tree = O.optimal_tree(e)[0]
    y = _run(emul, spec, shapes, False, 0, ins, out_shape=out_shape, generic=0)
    g = _run(emul, spec, shapes, False, 1, ins, dy=dy, generic=0)
    assert _rel(y, O.eval_pairwise(e, ins, tree)) <= 1e-5
    for a, b in zip(g, O.grads_pairwise(e, ins, tree, dy)):
        assert _rel(a, b) <= 1e-5
