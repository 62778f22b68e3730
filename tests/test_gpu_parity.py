"""GPU parity: the HIP path (through the C ABI) against the float64 oracle.

Reduced sizes compare Y and every gradient with the oracle's pairwise
evaluation along the same tree; full sizes compare with the oracle's dense
evaluation.  Every comparison (`_check`) applies two bars with the same
tolerance tol (1e-5 for float32, 2e-2 for bfloat16 inputs):

  * the whole tensor:   ||y - ref||_2 <= tol * ||ref||_2  (rel-L2), and
  * every element:      |y_i - ref_i| <= tol * max_j |ref_j|,

and prints the worst element's index.  For a correct result the largest
element error relative to max|ref| is about the rel-L2 error (both are set by
the rounding of the same sums), far below tol; a wrongly computed element
fails the second bar whenever its true value exceeds tol * max|ref|.
"""
import sys

import numpy as np
import pytest

import oracle as O
import workloads as W
from conftest import (CIRCULAR_CASES, EDGE_CASES, PAPER_SHAPES, STRIDED_CASES, load_layer_strings,
                      strides_of)

STRINGS = load_layer_strings()

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def P():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a HIP device")
    import paper_2401_03384_amd as P
    P.lib()
    return P


def _dev(a, bf16):
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return (t.to(torch.bfloat16) if bf16 else t).cuda()


def _host(t):
    return t.float().cpu().numpy().astype(np.float64)


def _rel(a, b):
    return float(np.linalg.norm((a - b).ravel()) / max(np.linalg.norm(b.ravel()), 1e-300))


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _check(what, got, ref, tol):
    """rel-L2 <= tol over the tensor and |got - ref| <= tol * max|ref| for
    every element; prints both and the worst element (NaN fails both)."""
    g = _host(got) if torch.is_tensor(got) else np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert g.shape == ref.shape, (what, g.shape, ref.shape)
    d = np.abs(g - ref)
    scale = max(float(np.abs(ref).max()), 1e-300)
    i = int(np.argmax(d)) if d.size else 0
    worst = float(d.ravel()[i]) / scale if d.size else 0.0
    rel = _rel(g, ref)
    idx = tuple(int(x) for x in np.unravel_index(i, ref.shape)) if d.size else ()
    _say(f"  {what}: rel-L2 {rel:.3e}  worst element {idx} |err|/max|ref| {worst:.3e}")
    assert rel <= tol, (what, "rel-L2", rel, tol)
    assert worst <= tol, (what, "element", idx, worst, tol)


def _check_all(name, y, y_ref, grads, g_ref, tol):
    _check(f"{name} Y", y, y_ref, tol)
    for i, (g, r) in enumerate(zip(grads, g_ref)):
        if g is not None:
            _check(f"{name} d{i}", g, r, tol)


PARITY = sorted(W.PARITY_WORKLOADS)


@pytest.mark.parametrize("generic", [False, True], ids=["default", "generic"])
@pytest.mark.parametrize("name", PARITY)
def test_parity_reduced(P, name, generic):
    w = W.PARITY_WORKLOADS[name]
    bf16 = w.dtype == "bf16"
    tol = 2e-2 if bf16 else 1e-5
    _say(f"case {name} generic={generic} shapes={w.shapes}")
    ins, dy = W.make_inputs(w)
    e = O.bind(O.parse(w.spec), w.shapes)
    tree = O.optimal_tree(e)[0]
    y_ref = O.eval_pairwise(e, ins, tree)
    plan = P.Plan(w.spec, w.shapes, w.dtype, flags=P.CE_FLAG_GENERIC_ONLY if generic else 0)
    xs = [_dev(a, bf16) for a in ins]
    y = plan.forward(xs)
    torch.cuda.synchronize()
    _check(f"{name} Y", y, y_ref, tol)
    if not w.backward:
        return
    g_ref = O.grads_pairwise(e, ins, tree, dy)
    grads = plan.backward(xs, _dev(dy, bf16))
    torch.cuda.synchronize()
    for i, (g, r) in enumerate(zip(grads, g_ref)):
        _check(f"{name} d{i}", g, r, tol)


@pytest.mark.parametrize("name", ["C2s", "C3s_f32", "C5bs"])
def test_deterministic(P, name):
    w = W.PARITY_WORKLOADS[name]
    bf16 = w.dtype == "bf16"
    ins, dy = W.make_inputs(w)
    plan = P.Plan(w.spec, w.shapes, w.dtype)
    xs = [_dev(a, bf16) for a in ins]
    d = _dev(dy, bf16)
    y1, y2 = plan.forward(xs), plan.forward(xs)
    g1, g2 = plan.backward(xs, d), plan.backward(xs, d)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
    for a, b in zip(g1, g2):
        assert torch.equal(a, b)


def test_partial_gradients(P):
    """NULL gradient entries are skipped; the others are unchanged."""
    w = W.PARITY_WORKLOADS["C2s"]
    ins, dy = W.make_inputs(w)
    plan = P.Plan(w.spec, w.shapes, w.dtype)
    xs = [_dev(a, False) for a in ins]
    d = _dev(dy, False)
    full = plan.backward(xs, d)
    part = plan.backward(xs, d, needs=[False, True, False, False, True])
    torch.cuda.synchronize()
    assert part[0] is None and part[2] is None
    assert torch.equal(part[1], full[1]) and torch.equal(part[4], full[4])


def test_autograd_function(P):
    w = W.PARITY_WORKLOADS["C2s"]
    ins, dy = W.make_inputs(w)
    xs = [_dev(a, False).requires_grad_(True) for a in ins]
    y = P.conv_einsum(w.spec, *xs)
    y.backward(_dev(dy, False))
    e = O.bind(O.parse(w.spec), w.shapes)
    g_ref = O.grads_dense(e, ins, dy)
    for i, (x, r) in enumerate(zip(xs, g_ref)):
        _check(f"autograd d{i}", x.grad, r, 1e-5)


FULL = ["C1", "C2", "C2_bf16", "C3", "C4", "C5a", "C5b"]


@pytest.mark.parametrize("name", FULL)
def test_parity_full_size(P, name):
    """Full-size layers against the oracle's dense evaluation (float64)."""
    w = W.WORKLOADS[name]
    bf16 = w.dtype == "bf16"
    tol = 2e-2 if bf16 else 1e-5
    _say(f"case {name} full size shapes={w.shapes}")
    ins, dy = W.make_inputs(w)
    e = O.bind(O.parse(w.spec), w.shapes)
    plan = P.Plan(w.spec, w.shapes, w.dtype)
    xs = [_dev(a, bf16) for a in ins]
    y = plan.forward(xs)
    torch.cuda.synchronize()
    _check(f"{name} Y", y, O.eval_dense(e, ins), tol)
    del y
    if not w.backward:
        return
    grads = plan.backward(xs, _dev(dy, bf16))
    torch.cuda.synchronize()
    g_ref = O.grads_dense(e, ins, dy)
    for i, (g, r) in enumerate(zip(grads, g_ref)):
        _check(f"{name} d{i}", g, r, tol)


@pytest.mark.parametrize("name", ["C2s", "C3s", "C4s", "C5as_f32", "C5bs"])
def test_saved_intermediates(P, name):
    """CE_FLAG_SAVE_INTERMEDIATES: the backward reads the intermediates the
    forward left in the shared workspace (no recompute) and matches the oracle."""
    w = W.PARITY_WORKLOADS[name]
    bf16 = w.dtype == "bf16"
    tol = 2e-2 if bf16 else 1e-5
    _say(f"case {name} saved intermediates shapes={w.shapes}")
    ins, dy = W.make_inputs(w)
    e = O.bind(O.parse(w.spec), w.shapes)
    tree = O.optimal_tree(e)[0]
    plan = P.Plan(w.spec, w.shapes, w.dtype, flags=P.CE_FLAG_SAVE_INTERMEDIATES)
    xs = [_dev(a, bf16) for a in ins]
    ws = plan.workspace(True, xs[0].device)
    y = plan.forward(xs, workspace=ws)
    grads = plan.backward(xs, _dev(dy, bf16), workspace=ws)
    torch.cuda.synchronize()
    _check_all(name, y, O.eval_pairwise(e, ins, tree), grads, O.grads_pairwise(e, ins, tree, dy), tol)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("name", sorted(PAPER_SHAPES))
def test_paper_layer_strings(P, name, dtype):
    """Every layer string the paper prints (CP, reshaped CP, Tucker, reshaped
    Tucker, tensor-train and -ring, block-term, hierarchical Tucker, separable
    and interleaved group convolutions (circular: h, w held by three
    operands), the Figure 1 sequence example (circular j), conv1d, grouped
    conv, mode convolution, contractions, outer and batch products) through
    the default plan, forward and all gradients, against the oracle."""
    spec = STRINGS[name][0]
    shapes = PAPER_SHAPES[name]
    bf16 = dtype == "bf16"
    tol = 2e-2 if bf16 else 1e-5
    _say(f"case {name} {dtype} {spec} shapes={shapes}")
    e = O.bind(O.parse(spec), shapes)
    plan = P.Plan(spec, shapes, dtype)
    rng = np.random.default_rng(7)
    ins = [rng.standard_normal(s) for s in shapes]
    if bf16:
        ins = [W.round_to_bf16(a.astype(np.float32)).astype(np.float64) for a in ins]
    else:
        ins = [a.astype(np.float32).astype(np.float64) for a in ins]
    out_shape = tuple(plan.out_shape)
    dy = rng.standard_normal(out_shape)
    dy = (W.round_to_bf16(dy.astype(np.float32)) if bf16 else dy.astype(np.float32)).astype(np.float64)
    tree = O.optimal_tree(e)[0]
    xs = [_dev(a, bf16) for a in ins]
    y = plan.forward(xs)
    grads = plan.backward(xs, _dev(dy, bf16))
    torch.cuda.synchronize()
    _check_all(name, y, O.eval_pairwise(e, ins, tree), grads, O.grads_pairwise(e, ins, tree, dy), tol)


@pytest.mark.parametrize("name", ["C4s", "C5as", "C5bs"])
def test_memory_limited_plan(P, name):
    """A cap just below the optimum's largest intermediate forces another
    order (the paper's memory/compute trade-off); it runs through the same
    kernels and matches the oracle along the oracle's limited tree."""
    w = W.PARITY_WORKLOADS[name]
    bf16 = w.dtype == "bf16"
    tol = 2e-2 if bf16 else 1e-5
    ins, dy = W.make_inputs(w)
    e = O.bind(O.parse(w.spec), w.shapes)
    cap = O.max_intermediate(e, O.optimal_tree(e)[0]) - 1
    tree, _ = O.optimal_tree(e, max_elements=cap)
    assert tree is not None
    _say(f"case {name} limited to {cap} elements, tree {tree}")
    plan = P.Plan(w.spec, w.shapes, w.dtype, max_elements=cap)
    xs = [_dev(a, bf16) for a in ins]
    y = plan.forward(xs)
    grads = plan.backward(xs, _dev(dy, bf16))
    torch.cuda.synchronize()
    _check_all(name, y, O.eval_pairwise(e, ins, tree), grads, O.grads_pairwise(e, ins, tree, dy), tol)


@pytest.mark.parametrize("name", ["C1", "C2s", "C3s", "C5as"])
def test_graph_replay(P, name):
    """Forward + backward captured as a HIP graph: three replays, with eager
    work and synchronisations in between, each equal (bit for bit: the
    kernels are deterministic) to the eager result."""
    w = W.PARITY_WORKLOADS[name]
    bf16 = w.dtype == "bf16"
    _say(f"case {name} graph replay")
    ins, dy = W.make_inputs(w)
    plan = P.Plan(w.spec, w.shapes, w.dtype)
    xs = [_dev(a, bf16) for a in ins]
    d = _dev(dy, bf16)
    y_ref = plan.forward(xs)
    g_ref = plan.backward(xs, d)
    torch.cuda.synchronize()
    step = P.GraphStep(plan, xs, d)
    for k in range(3):
        step.out.zero_()
        for g in step.grads:
            g.zero_()
        step.replay()
        torch.cuda.synchronize()
        assert torch.equal(step.out, y_ref), (name, k)
        for i, (g, r) in enumerate(zip(step.grads, g_ref)):
            assert torch.equal(g, r), (name, k, i)
        # eager work between replays
        plan.forward(xs)
        torch.cuda.synchronize()


def _random_case(spec, shapes, dtype, feat=0, seed=7, strides=None, circular=()):
    """Seeded N(0,1) operands and dY for a small case, rounded to the storage
    type; the oracle expression bound with the same feature operand."""
    bf16 = dtype == "bf16"
    e = O.bind(O.parse(spec), shapes, feature_operand=feat, strides=strides, circular=circular)
    rng = np.random.default_rng(seed)
    rnd = (lambda a: W.round_to_bf16(a.astype(np.float32))) if bf16 else (lambda a: a.astype(np.float32))
    ins = [rnd(rng.standard_normal(s)).astype(np.float64) for s in shapes]
    out_shape = tuple(e.out_sizes[l] for l in e.output)
    dy = rnd(rng.standard_normal(out_shape)).astype(np.float64)
    return e, ins, dy


@pytest.mark.parametrize("generic", [False, True], ids=["default", "generic"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("name", sorted(EDGE_CASES))
def test_edge_cases(P, name, dtype, generic):
    """Pre-summed labels, single operands, the feature operand second, equal
    feature / filter sizes with a designated feature operand, even filters:
    forward and every gradient against the oracle along the same tree."""
    spec, shapes, feat = EDGE_CASES[name]
    bf16 = dtype == "bf16"
    tol = 2e-2 if bf16 else 1e-5
    _say(f"case {name} {dtype} generic={generic} {spec} shapes={shapes} feature={feat}")
    e, ins, dy = _random_case(spec, shapes, dtype, feat)
    plan = P.Plan(spec, shapes, dtype, feature_operand=feat,
                  flags=P.CE_FLAG_GENERIC_ONLY if generic else 0)
    assert tuple(plan.out_shape) == dy.shape
    tree = O.optimal_tree(e)[0]
    xs = [_dev(a, bf16) for a in ins]
    y = plan.forward(xs)
    grads = plan.backward(xs, _dev(dy, bf16))
    torch.cuda.synchronize()
    _check_all(name, y, O.eval_pairwise(e, ins, tree), grads, O.grads_pairwise(e, ins, tree, dy), tol)


LTR = ["C2s", "C2s_bf16", "C3s", "C4s", "C5bs", "C5as_f32"]


@pytest.mark.parametrize("name", LTR)
def test_left_to_right_plan(P, name):
    """The paper's baseline order (((X, A), B), ...) on the same kernels,
    against the oracle evaluated along the left-to-right tree."""
    w = W.PARITY_WORKLOADS[name]
    bf16 = w.dtype == "bf16"
    tol = 2e-2 if bf16 else 1e-5
    n = len(w.shapes)
    path = [(0, 1)] + [(0, n - 1 - k) for k in range(1, n - 1)]
    _say(f"case {name} left-to-right path {path}")
    ins, dy = W.make_inputs(w)
    e = O.bind(O.parse(w.spec), w.shapes)
    tree = O.left_to_right_tree(n)
    plan = P.Plan(w.spec, w.shapes, w.dtype, path=path)
    assert [(a, b) for a, b, _ in plan.steps][0] == (1, 2)
    xs = [_dev(a, bf16) for a in ins]
    y = plan.forward(xs)
    grads = plan.backward(xs, _dev(dy, bf16))
    torch.cuda.synchronize()
    _check_all(name, y, O.eval_pairwise(e, ins, tree), grads, O.grads_pairwise(e, ins, tree, dy), tol)


@pytest.mark.parametrize("name,ltr", [("C2s", True), ("C2s_bf16", True), ("C4s", False),
                                      ("C3c5", False), ("C5as_f32", True)])
def test_wide_offsets(P, name, ltr):
    """CE_FLAG_WIDE_OFFSETS: the general contraction kernel's 64-bit offset
    path (used for operands beyond 2 GiB) at small sizes, against the oracle
    and bit-equal to the 32-bit path."""
    w = W.PARITY_WORKLOADS[name]
    bf16 = w.dtype == "bf16"
    tol = 2e-2 if bf16 else 1e-5
    n = len(w.shapes)
    path = [(0, 1)] + [(0, n - 1 - k) for k in range(1, n - 1)] if ltr else None
    tree = O.left_to_right_tree(n) if ltr else None
    ins, dy = W.make_inputs(w)
    e = O.bind(O.parse(w.spec), w.shapes)
    if tree is None:
        tree = O.optimal_tree(e)[0]
    flags = P.CE_FLAG_NO_FUSION
    wide = P.Plan(w.spec, w.shapes, w.dtype, path=path, flags=flags | P.CE_FLAG_WIDE_OFFSETS)
    narrow = P.Plan(w.spec, w.shapes, w.dtype, path=path, flags=flags)
    assert "tc_gemm" in wide.describe(), "no launch of the general contraction kernel"
    _say(f"case {name} wide offsets, tree {tree}")
    xs = [_dev(a, bf16) for a in ins]
    d = _dev(dy, bf16)
    y = wide.forward(xs)
    grads = wide.backward(xs, d)
    y2 = narrow.forward(xs)
    grads2 = narrow.backward(xs, d)
    torch.cuda.synchronize()
    _check_all(name, y, O.eval_pairwise(e, ins, tree), grads, O.grads_pairwise(e, ins, tree, dy), tol)
    assert torch.equal(y, y2)
    for a, b in zip(grads, grads2):
        assert torch.equal(a, b)


@pytest.mark.parametrize("name,nofuse", [("C2s", True), ("C3s", False), ("C4s", False),
                                         ("C5bs", True), ("C5as_f32", False)])
def test_save_budget(P, name, nofuse):
    """Checkpointing under a save budget (Section 3.3): the forward keeps the
    chosen intermediates in the workspace, the backward reads them and
    recomputes the rest; against the oracle."""
    w = W.PARITY_WORKLOADS[name]
    bf16 = w.dtype == "bf16"
    tol = 2e-2 if bf16 else 1e-5
    ins, dy = W.make_inputs(w)
    e = O.bind(O.parse(w.spec), w.shapes)
    tree = O.optimal_tree(e)[0]
    total = O.checkpoint_choice(e, tree, 10 ** 18, 2 if bf16 else 4)[1]
    flags = P.CE_FLAG_NO_FUSION if nofuse else 0
    plan = P.Plan(w.spec, w.shapes, w.dtype, flags=flags, save_budget=total // 2)
    _say(f"case {name} save budget {total // 2} of {total} B: kept steps {plan.saved_steps:#x}, "
         f"{plan.saved_bytes} B, recompute {plan.recompute_macs} MACs")
    assert plan.saved_steps != 0
    xs = [_dev(a, bf16) for a in ins]
    ws = plan.workspace(True, xs[0].device)
    y = plan.forward(xs, workspace=ws)
    grads = plan.backward(xs, _dev(dy, bf16), workspace=ws)
    torch.cuda.synchronize()
    _check_all(name, y, O.eval_pairwise(e, ins, tree), grads, O.grads_pairwise(e, ins, tree, dy), tol)


@pytest.mark.parametrize("name", ["rtt_conv", "tr_conv"])
def test_cost_capped_plan(P, name):
    """A per-step cost cap one below the optimum's largest step (Section 3.2,
    Figure 2) forces another order; it runs on the same kernels and matches
    the oracle along the oracle's capped tree."""
    spec, shapes = STRINGS[name][0], PAPER_SHAPES[name]
    e, ins, dy = _random_case(spec, shapes, "f32")
    t0 = O.optimal_tree(e)[0]
    cap = max(O.step_costs(e, t0)) - 1
    tree, _ = O.optimal_tree(e, max_step_cost=cap)
    assert tree is not None and tree != t0
    plan = P.Plan(spec, shapes, "f32", max_step_cost=cap)
    _say(f"case {name} step cost cap {cap}: tree {tree}")
    xs = [_dev(a, False) for a in ins]
    y = plan.forward(xs)
    grads = plan.backward(xs, _dev(dy, False))
    torch.cuda.synchronize()
    _check_all(name, y, O.eval_pairwise(e, ins, tree), grads, O.grads_pairwise(e, ins, tree, dy), 1e-5)


@pytest.mark.parametrize("generic", [False, True], ids=["default", "generic"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("name", sorted(STRIDED_CASES))
def test_strided(P, name, dtype, generic):
    """Strided convolutions (Appendix B varieties): forward, and the backward
    whose transposed convolutions run as stride-1 phases on views of the
    gradient and the filter; against the oracle."""
    spec, shapes, st = STRIDED_CASES[name]
    strides = strides_of(st)
    bf16 = dtype == "bf16"
    tol = 2e-2 if bf16 else 1e-5
    _say(f"case {name} {dtype} generic={generic} {spec} shapes={shapes} strides={strides}")
    e, ins, dy = _random_case(spec, shapes, dtype, strides=strides)
    plan = P.Plan(spec, shapes, dtype, strides=strides,
                  flags=P.CE_FLAG_GENERIC_ONLY if generic else 0)
    assert tuple(plan.out_shape) == dy.shape
    tree = O.optimal_tree(e)[0]
    xs = [_dev(a, bf16) for a in ins]
    y = plan.forward(xs)
    grads = plan.backward(xs, _dev(dy, bf16))
    torch.cuda.synchronize()
    _check_all(name, y, O.eval_pairwise(e, ins, tree), grads, O.grads_pairwise(e, ins, tree, dy), tol)


@pytest.mark.parametrize("order", ["optimal", "ltr"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("name", [r[0] for r in W.RESNET34_CONVS])
def test_resnet34_cp_layers(P, name, dtype, order):
    """The ResNet-34 convolutions as CP layers (7x7 stem, 3x3 and strided
    3x3, strided 1x1 shortcuts) at reduced size (channels and input / 8),
    the planned and the left-to-right order, against the oracle along the
    same tree."""
    w, strides = W.resnet34_cp_layer(name, batch=2, scale=8, dtype=dtype)
    bf16 = dtype == "bf16"
    tol = 2e-2 if bf16 else 1e-5
    ins, dy = W.make_inputs(w)
    e = O.bind(O.parse(w.spec), w.shapes, strides=strides)
    path = [(0, 1), (0, 3), (0, 2), (0, 1)] if order == "ltr" else None
    tree = O.left_to_right_tree(5) if order == "ltr" else O.optimal_tree(e)[0]
    _say(f"case {w.name} {dtype} {order} shapes={w.shapes} strides={strides} tree {tree}")
    plan = P.Plan(w.spec, w.shapes, dtype, strides=strides, path=path)
    xs = [_dev(a, bf16) for a in ins]
    y = plan.forward(xs)
    grads = plan.backward(xs, _dev(dy, bf16))
    torch.cuda.synchronize()
    _check_all(w.name, y, O.eval_pairwise(e, ins, tree), grads, O.grads_pairwise(e, ins, tree, dy), tol)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("name", sorted(CIRCULAR_CASES))
def test_circular(P, name, dtype):
    """Circular convolutions (Appendix B: commutative, the only kind for a
    label held by three or more operands), two-, three- and four-way, through
    the planned order and every other tree's first steps, against the oracle
    along the same tree."""
    spec, shapes, circ = CIRCULAR_CASES[name]
    bf16 = dtype == "bf16"
    tol = 2e-2 if bf16 else 1e-5
    e, ins, dy = _random_case(spec, shapes, dtype, circular=circ)
    n = len(shapes)
    paths = [None, [(0, 1)] + [(0, n - 1 - k) for k in range(1, n - 1)]]
    trees = [O.optimal_tree(e)[0], O.left_to_right_tree(n)]
    xs = [_dev(a, bf16) for a in ins]
    for path, tree in zip(paths, trees):
        _say(f"case {name} {dtype} {spec} shapes={shapes} tree {tree}")
        plan = P.Plan(spec, shapes, dtype, path=path, circular=circ)
        assert tuple(plan.out_shape) == dy.shape
        y = plan.forward(xs)
        grads = plan.backward(xs, _dev(dy, bf16))
        torch.cuda.synchronize()
        _check_all(name, y, O.eval_pairwise(e, ins, tree), grads,
                   O.grads_pairwise(e, ins, tree, dy), tol)
