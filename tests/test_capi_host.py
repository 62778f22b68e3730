"""C-ABI host-side tests (no GPU): the library loads and exports every symbol
include/convein.h declares; the C++ planner reproduces the oracle's brute-force
plan (tree, per-step multiplications, totals, both cost modes) on every
workload, every printed layer string and random expressions; error paths
return their status codes before any device call."""
import ctypes as C
import os
import random
import re

import pytest

import oracle as O
import workloads as W
from conftest import PAPER_SHAPES, ROOT, load_layer_strings

B = pytest.importorskip("paper_2401_03384_amd.binding")

STRINGS = load_layer_strings()


def _mask(t):
    return sum(1 << i for i in O.leaves(t))


def _oracle_steps(e, tree, mode="fwd"):
    steps = O.post_order_steps(tree)
    costs = O.step_costs(e, tree, "fwd")
    return [(_mask(a), _mask(b), c) for (a, b), c in zip(steps, costs)]


def _plan(spec, shapes, mode=B.CE_COST_FWD, dtype=B.CE_F32, feature=0):
    e = B.ce_expr_parse(spec, shapes)
    try:
        if feature:
            B.ce_expr_set_feature(e, feature)
        return B.ce_plan_create(e, mode, dtype, 0)
    finally:
        B.ce_expr_destroy(e)


def _steps(p):
    return [B.ce_plan_step(p, i) for i in range(B.ce_plan_num_steps(p))]


def test_every_declared_symbol_is_exported():
    header = open(os.path.join(ROOT, "include", "convein.h")).read()
    declared = set(re.findall(r"^(?:ce_status|void|const char\*)\s+(ce_[a-z_]+)\s*\(", header,
                              re.M))
    L = B.lib()
    for name in declared:
        assert hasattr(L, name), name
        assert isinstance(getattr(L, name), C._CFuncPtr)
    assert declared == set(B.EXPORTS)
    assert "gfx950" in B.ce_version()


def _compare(spec, shapes, feature=0):
    e = O.bind(O.parse(spec), shapes, feature_operand=feature)
    for mode, cmode in (("fwd", B.CE_COST_FWD), ("train_paper", B.CE_COST_TRAIN_PAPER)):
        tree, cost = O.optimal_tree(e, mode)
        p = _plan(spec, shapes, cmode, feature=feature)
        try:
            assert _steps(p) == _oracle_steps(e, tree), (spec, mode)
            total, fwd = B.ce_plan_cost(p)
            assert total == cost
            assert fwd == O.tree_cost(e, tree, "fwd")
            assert B.ce_plan_left_to_right_cost(p) == O.tree_cost(e, O.left_to_right_tree(e.n), mode)
        finally:
            B.ce_plan_destroy(p)


@pytest.mark.parametrize("name", sorted(set(W.WORKLOADS) | set(W.PARITY_WORKLOADS)))
def test_planner_matches_oracle_on_workloads(name):
    w = W.WORKLOADS.get(name) or W.PARITY_WORKLOADS[name]
    _compare(w.spec, w.shapes)




@pytest.mark.parametrize("name", sorted(PAPER_SHAPES))
def test_planner_matches_oracle_on_paper_strings(name):
    _compare(STRINGS[name][0], PAPER_SHAPES[name])


def _random_expr(rnd):
    n = rnd.randint(2, 6)
    pool = "abcdefghijk"
    nl = rnd.randint(2, 8)
    labels = list(pool[:nl])
    size = {l: rnd.randint(1, 4) for l in labels}
    ops = [[] for _ in range(n)]
    for l in labels:
        k = rnd.choice([1, 1, 2, 2, 2, 3])
        for i in rnd.sample(range(n), min(k, n)):
            ops[i].append(l)
    for i in range(n):
        if not ops[i]:
            ops[i].append(rnd.choice(labels))
        rnd.shuffle(ops[i])
    present = sorted({l for t in ops for l in t})
    holders = {l: [i for i in range(n) if l in ops[i]] for l in present}
    conv = [l for l in present if len(holders[l]) >= 2 and rnd.random() < 0.3]
    out = [l for l in present if l in conv or rnd.random() < 0.4]
    rnd.shuffle(out)
    shapes = []
    for i in range(n):
        shp = []
        for l in ops[i]:
            if l in conv:
                shp.append(rnd.randint(1, 6))
            else:
                shp.append(size[l])
        shapes.append(tuple(shp))
    spec = ",".join("".join(t) for t in ops) + "->" + "".join(out)
    if conv:
        spec += "|" + "".join(conv)
    return spec, shapes, rnd.randrange(n)


@pytest.mark.parametrize("seed", range(40))
def test_planner_matches_oracle_on_random_expressions(seed):
    # 40 x 25 = 1000 random expressions of 2 to 6 operands
    rnd = random.Random(1000 + seed)
    for _ in range(25):
        spec, shapes, feat = _random_expr(rnd)
        _compare(spec, shapes, feature=feat)


# The tensor-train layer with every core split into a chain of two-way and
# three-way factors: eight operands, 135,135 binary trees (the planner's
# stress case; the C4 sizes, TT ranks 16).
SPLIT_TT = ("b(s1)(s2)(s3)hw,(s1)(a1),(a1)(s2)(a2),(a2)(s3)(a3),(a3)hw(a4),(a4)(t1)(a5),(a5)(t2)(a6),(a6)(t3)"
            "->b(t1)(t2)(t3)hw|hw",
            [(64, 4, 8, 8, 28, 28), (4, 16), (16, 8, 16), (16, 8, 16), (16, 3, 3, 16), (16, 4, 16),
             (16, 8, 16), (16, 8)])


def test_planner_eight_operand_split_chain():
    spec, shapes = SPLIT_TT
    e = O.bind(O.parse(spec), shapes)
    best, cost, ties = O.optimal_tree(e, return_all=True)
    assert len(ties) == 1 and cost == 526802944   # unique optimum
    assert O.count_trees(8) == 135135
    _compare(spec, shapes)


def test_user_path_and_left_to_right():
    w = W.WORKLOADS["C2"]
    e = B.ce_expr_parse(w.spec, w.shapes)
    # merged tensors are appended: left-to-right pairs the last entry with position 0
    p = B.ce_plan_create_with_path(e, [(0, 1), (0, 3), (0, 2), (0, 1)], B.CE_F32, 0)
    B.ce_expr_destroy(e)
    oe = O.bind(O.parse(w.spec), w.shapes)
    ltr = O.left_to_right_tree(5)
    assert _steps(p) == _oracle_steps(oe, ltr)
    assert B.ce_plan_cost(p)[0] == O.tree_cost(oe, ltr) == 6576668672
    # workspace of the left-to-right plan holds the 822M-element intermediate
    assert B.ce_plan_workspace_size(p, 0) >= 128 * 32 * 64 * 56 * 56 * 4
    B.ce_plan_destroy(p)


def test_workspace_covers_live_intermediates():
    w = W.WORKLOADS["C2"]
    e = B.ce_expr_parse(w.spec, w.shapes)
    p = B.ce_plan_create(e, B.CE_COST_FWD, B.CE_F32, B.CE_FLAG_NO_FUSION)
    B.ce_expr_destroy(e)
    fwd, bwd = B.ce_plan_workspace_size(p, 0), B.ce_plan_workspace_size(p, 1)
    inter = 128 * 32 * 56 * 56 * 4
    assert fwd >= 2 * inter          # two intermediates are live at once
    assert bwd >= 3 * inter          # three recomputed values, plus gradients
    B.ce_plan_destroy(p)


def test_fused_chain_keeps_intermediates_on_chip():
    """The fused CP chain needs no intermediate in HBM: the forward takes no
    workspace, the backward only the per-block factor-gradient partials."""
    w = W.WORKLOADS["C2"]
    p = _plan(w.spec, w.shapes)
    assert "fused CP chain backward" in B.ce_plan_describe(p)
    fwd, bwd = B.ce_plan_workspace_size(p, 0), B.ce_plan_workspace_size(p, 1)
    assert fwd == 0
    inter = 128 * 32 * 56 * 56 * 4
    assert 0 < bwd < inter // 4
    B.ce_plan_destroy(p)


@pytest.mark.parametrize("name,fused", [("C5a", True), ("C5b", True), ("C5as", True), ("C5bs", True),
                                        ("C5bt2", True), ("C5bt3", True), ("C5as_f32", False),
                                        ("C5cs", False)])
def test_fused_rcp_forward(name, fused):
    """Reshaped-CP layers of a compiled instantiation run their whole forward
    as one launch with no workspace; other shapes and float32 stay unfused."""
    w = W.WORKLOADS.get(name) or W.PARITY_WORKLOADS[name]
    p = _plan(w.spec, w.shapes, dtype=B.CE_BF16 if w.dtype == "bf16" else B.CE_F32)
    text = B.ce_plan_describe(p)
    fwd = [l for l in text.splitlines() if l.startswith("  fwd ")]
    if fused:
        assert len(fwd) == 1 and "fused RCP chain" in fwd[0]
        assert B.ce_plan_workspace_size(p, 0) == 0
    else:
        assert not any("fused RCP" in l for l in fwd)
    B.ce_plan_destroy(p)


@pytest.mark.parametrize("spec,shapes,status", [
    ("bshw,tshw", [(1, 2, 3, 3), (1, 2, 3, 3)], B.CE_ERR_PARSE),
    ("bssw,tshw->bthw|hw", [(1, 2, 2, 3), (1, 2, 3, 3)], B.CE_ERR_PARSE),
    ("bshw,tshw->bthwx", [(1, 2, 3, 3), (1, 2, 3, 3)], B.CE_ERR_PARSE),
    ("bshw,tshw->bt|hw", [(1, 2, 3, 3), (1, 2, 3, 3)], B.CE_ERR_PARSE),
    ("bs(h,tshw->bthw", [(1, 2, 3), (1, 2, 3, 3)], B.CE_ERR_PARSE),
    ("bshw,tshw->bthw|hw", [(1, 2, 3, 3), (1, 5, 3, 3)], B.CE_ERR_SHAPE),
    ("bshw,tshw->bthw|hw", [(1, 2, 3), (1, 2, 3, 3)], B.CE_ERR_SHAPE),
    ("bshw,tshw->bthw|hw", [(1, 2, 3, 3)], B.CE_ERR_SHAPE),
    ("bshw,tshw->bthw|hw", [(1, 0, 3, 3), (1, 0, 3, 3)], B.CE_ERR_SHAPE),
])
def test_errors_are_reported(spec, shapes, status):
    with pytest.raises(B.CeError) as ex:
        B.ce_expr_parse(spec, shapes)
    assert ex.value.status == status
    assert B.ce_last_error()


def test_cost_overflow_is_reported():
    big = 1 << 30
    e = B.ce_expr_parse("ab,bc,cd->ad", [(big, big), (big, big), (big, big)])
    with pytest.raises(B.CeError) as ex:
        B.ce_plan_create(e, B.CE_COST_FWD, B.CE_F32, 0)
    assert ex.value.status == B.CE_ERR_OVERFLOW
    B.ce_expr_destroy(e)


def test_execution_errors_before_any_device_call():
    """Validation runs before any launch: these return without touching a GPU."""
    L = B.lib()
    fake = C.c_void_p(0x1000)
    ins = (C.c_void_p * 2)(fake, fake)
    # a circular plan with a too small workspace
    p = _plan("bfhw,fghw,sghw->bshw|hw", [(1, 2, 5, 5), (2, 3, 3, 3), (4, 3, 3, 3)])
    ins3 = (C.c_void_p * 3)(fake, fake, fake)
    assert B.ce_plan_workspace_size(p, 0) > 0
    assert L.ce_forward(p, ins3, fake, fake, 0, None) == B.CE_ERR_WORKSPACE
    B.ce_plan_destroy(p)
    p = _plan("bshw,tshw->bthw|hw", [(2, 3, 8, 8), (4, 3, 3, 3)])
    assert L.ce_forward(p, ins, None, None, 0, None) == B.CE_ERR_ARG
    assert L.ce_forward(None, ins, fake, None, 0, None) == B.CE_ERR_ARG
    null_in = (C.c_void_p * 2)(fake, None)
    assert L.ce_forward(p, null_in, fake, None, 0, None) == B.CE_ERR_ARG
    din = (C.c_void_p * 2)(None, None)
    assert L.ce_backward(p, ins, None, din, None, 0, None) == B.CE_ERR_ARG
    B.ce_plan_destroy(p)
    # a plan with intermediates (unfused): workspace too small / misaligned
    w = W.PARITY_WORKLOADS["C2s"]
    e = B.ce_expr_parse(w.spec, w.shapes)
    p = B.ce_plan_create(e, B.CE_COST_FWD, B.CE_F32, B.CE_FLAG_NO_FUSION)
    B.ce_expr_destroy(e)
    assert B.ce_plan_workspace_size(p, 0) > 0
    ins5 = (C.c_void_p * 5)(*([fake] * 5))
    need = B.ce_plan_workspace_size(p, 0)
    assert L.ce_forward(p, ins5, fake, fake, need - 1, None) == B.CE_ERR_WORKSPACE
    assert L.ce_forward(p, ins5, fake, C.c_void_p(0x1008), need, None) == B.CE_ERR_WORKSPACE
    assert L.ce_forward(p, ins5, fake, None, need, None) == B.CE_ERR_WORKSPACE
    din5 = (C.c_void_p * 5)(*([fake] * 5))
    needb = B.ce_plan_workspace_size(p, 1)
    assert L.ce_backward(p, ins5, fake, din5, fake, needb - 1, None) == B.CE_ERR_WORKSPACE
    # no gradient wanted: nothing to do, OK without launching
    none5 = (C.c_void_p * 5)(*([None] * 5))
    assert L.ce_backward(p, ins5, fake, none5, fake, needb, None) == B.CE_OK
    B.ce_plan_destroy(p)


def test_bad_path_rejected():
    e = B.ce_expr_parse("ab,bc,cd->ad", [(2, 3), (3, 4), (4, 5)])
    with pytest.raises(B.CeError) as ex:
        B.ce_plan_create_with_path(e, [(0, 0), (0, 1)], B.CE_F32, 0)
    assert ex.value.status == B.CE_ERR_ARG
    with pytest.raises(B.CeError):
        B.ce_plan_create_with_path(e, [(0, 1)], B.CE_F32, 0)
    B.ce_expr_destroy(e)


def test_feature_operand_designation():
    # equal sizes: the designated operand is the feature side
    spec, shapes = "bsh,tsh->bth|h", [(2, 3, 5), (4, 3, 5)]
    for feat in (0, 1):
        e = B.ce_expr_parse(spec, shapes)
        B.ce_expr_set_feature(e, feat)
        assert B.ce_expr_output_shape(e) == (2, 4, 5)
        p = B.ce_plan_create(e, B.CE_COST_TRAIN_PAPER, B.CE_F32, 0)
        oe = O.bind(O.parse(spec), shapes, feature_operand=feat)
        assert B.ce_plan_cost(p)[0] == O.tree_cost(oe, (0, 1), "train_paper")
        B.ce_plan_destroy(p)
        B.ce_expr_destroy(e)


def test_saved_intermediates_plan():
    """CE_FLAG_SAVE_INTERMEDIATES: no recompute launches in an unfused
    backward, the backward workspace covers the forward's; fused chains are
    unchanged."""
    w = W.WORKLOADS["C4"]
    e = B.ce_expr_parse(w.spec, w.shapes)
    p0 = B.ce_plan_create(e, B.CE_COST_FWD, B.CE_F32, 0)
    p1 = B.ce_plan_create(e, B.CE_COST_FWD, B.CE_F32, B.CE_FLAG_SAVE_INTERMEDIATES)
    B.ce_expr_destroy(e)
    assert "recompute" in B.ce_plan_describe(p0)
    assert "recompute" not in B.ce_plan_describe(p1)
    assert B.ce_plan_workspace_size(p1, 1) >= B.ce_plan_workspace_size(p1, 0) > 0
    B.ce_plan_destroy(p0)
    B.ce_plan_destroy(p1)
    w = W.WORKLOADS["C2"]
    e = B.ce_expr_parse(w.spec, w.shapes)
    p2 = B.ce_plan_create(e, B.CE_COST_FWD, B.CE_F32, B.CE_FLAG_SAVE_INTERMEDIATES)
    B.ce_expr_destroy(e)
    assert "fused CP chain backward" in B.ce_plan_describe(p2)
    assert B.ce_plan_workspace_size(p2, 0) == 0
    B.ce_plan_destroy(p2)


def test_set_conv():
    """Padding of a convolved label: zero 'same' or circular on a two-way
    label, circular only on a multi-way label; unknown paddings, unknown or
    non-convolved labels are argument errors."""
    e = B.ce_expr_parse("bshw,sthw->bthw|hw", [(1, 2, 5, 5), (2, 3, 3, 3)])
    try:
        B.ce_expr_set_conv(e, "h", B.CE_PAD_SAME_ZERO)
        B.ce_expr_set_conv(e, "w", B.CE_PAD_CIRCULAR)
        for label, pad, status in (("w", 7, B.CE_ERR_ARG), ("s", 0, B.CE_ERR_ARG),
                                   ("z", 0, B.CE_ERR_ARG)):
            with pytest.raises(B.CeError) as ex:
                B.ce_expr_set_conv(e, label, pad)
            assert ex.value.status == status
        with pytest.raises(B.CeError) as ex:
            B.ce_expr_set_stride(e, "w", 2)
            B.ce_plan_destroy(B.ce_plan_create(e, B.CE_COST_FWD, B.CE_F32, 0))
        assert ex.value.status == B.CE_ERR_UNSUPPORTED
    finally:
        B.ce_expr_destroy(e)
    e = B.ce_expr_parse("bfhw,fghw,sghw->bshw|hw", [(1, 2, 5, 5), (2, 3, 3, 3), (4, 3, 3, 3)])
    try:
        B.ce_expr_set_conv(e, "h", B.CE_PAD_CIRCULAR)
        with pytest.raises(B.CeError) as ex:
            B.ce_expr_set_conv(e, "w", B.CE_PAD_SAME_ZERO)
        assert ex.value.status == B.CE_ERR_UNSUPPORTED
    finally:
        B.ce_expr_destroy(e)


def _compare_limited(spec, shapes, limits):
    """ce_plan_create_limited == the oracle's memory-limited search (tree,
    per-step MACs, cost), or both infeasible."""
    e = O.bind(O.parse(spec), shapes)
    for cap in limits:
        tree, cost = O.optimal_tree(e, "fwd", max_elements=cap)
        ex = B.ce_expr_parse(spec, shapes)
        try:
            if tree is None:
                with pytest.raises(B.CeError) as err:
                    B.ce_plan_create_limited(ex, B.CE_COST_FWD, B.CE_F32, 0, cap)
                assert err.value.status == B.CE_ERR_UNSUPPORTED
                continue
            p = B.ce_plan_create_limited(ex, B.CE_COST_FWD, B.CE_F32, 0, cap)
        finally:
            B.ce_expr_destroy(ex)
        try:
            assert _steps(p) == _oracle_steps(e, tree), (spec, cap)
            assert B.ce_plan_cost(p)[0] == cost
        finally:
            B.ce_plan_destroy(p)


def _limits_for(e):
    """Caps around the largest intermediates of the unconstrained optimum and
    of the left-to-right tree (so both feasible and infeasible caps occur)."""
    t, _ = O.optimal_tree(e)
    m = O.max_intermediate(e, t)
    l = O.max_intermediate(e, O.left_to_right_tree(e.n))
    return sorted({max(m, 1), max(m - 1, 1), max(m // 2, 1), max(l, 1), max(l - 1, 1), 1})


@pytest.mark.parametrize("name", sorted(set(W.WORKLOADS) | {"C2s", "C3s", "C4s", "C5as"}))
def test_limited_planner_matches_oracle_on_workloads(name):
    w = W.WORKLOADS.get(name) or W.PARITY_WORKLOADS[name]
    _compare_limited(w.spec, w.shapes, _limits_for(O.bind(O.parse(w.spec), w.shapes)))


@pytest.mark.parametrize("seed", range(20))
def test_limited_planner_matches_oracle_on_random_expressions(seed):
    rnd = random.Random(5000 + seed)
    for _ in range(4):
        spec, shapes, _ = _random_expr(rnd)
        e = O.bind(O.parse(spec), shapes)
        if e.n > 6 or any(len(e.holders(l)) > 2 for l in e.conv):
            continue
        _compare_limited(spec, shapes, _limits_for(e))


@pytest.mark.parametrize("name,steps", [
    ("C3", ["step 1 fwd", "step 1 recompute", "step 1 grad lhs"]),
    ("C3s_f32", []),   # fp32 with 64 contracted channels: the general contraction is faster
    ("C3p5", ["step 2 fwd"]),
    ("C4", ["step 3 grad lhs"]),
    ("C3t", []),   # 16 output channels: the plane kernel, not MFMA tiles
])
def test_conv_contraction_kernel_selected(name, steps):
    """Steps that convolve and contract one channel index with more than 16
    output channels (and, in fp32, at most 8 contracted channels) run on the
    MFMA conv-contraction kernel (cconv, or its register-filter form cconv_r
    for fp32 with at most 9 taps), both forward and input gradient; the
    filter gradient does not."""
    w = W.WORKLOADS.get(name) or W.PARITY_WORKLOADS.get(name) or W.tucker2_layer(
        "C3t", 2, 32, 24, 7, 9, 8, 16, 3, "bf16", 21)
    p = _plan(w.spec, w.shapes, dtype=B.CE_BF16 if w.dtype == "bf16" else B.CE_F32)
    text = B.ce_plan_describe(p)
    B.ce_plan_destroy(p)
    on36 = [l for l in text.splitlines() if "cconv<" in l or "cconv_r<" in l]
    for s in steps:
        assert any(s in l for l in on36), (name, s, text)
    assert len(on36) == len(steps), (name, on36)
    assert not any("grad rhs" in l for l in on36)


def test_noalloc_backward_rejects_before_any_launch():
    """ce_backward_noalloc's checks (no device work happens on these paths):
    a backward workspace beyond CE_NOALLOC_WORKSPACE_BYTES, a plan that saves
    intermediates, NULL arguments."""
    w = W.WORKLOADS["C4"]
    p = _plan(w.spec, w.shapes)
    assert B.ce_plan_workspace_size(p, 1) > B.CE_NOALLOC_WORKSPACE_BYTES
    fake = [0x1000 * (i + 1) for i in range(len(w.shapes))]
    with pytest.raises(B.CeError) as ex:
        B.ce_backward_noalloc(p, fake, 0x9000, fake, 0)
    assert ex.value.status == B.CE_ERR_WORKSPACE
    B.ce_plan_destroy(p)
    w = W.PARITY_WORKLOADS["C2s"]
    e = B.ce_expr_parse(w.spec, w.shapes)
    p = B.ce_plan_create(e, B.CE_COST_FWD, B.CE_F32, B.CE_FLAG_SAVE_INTERMEDIATES | B.CE_FLAG_NO_FUSION)
    B.ce_expr_destroy(e)
    with pytest.raises(B.CeError) as ex:
        B.ce_backward_noalloc(p, fake, 0x9000, fake, 0)
    assert ex.value.status == B.CE_ERR_UNSUPPORTED
    with pytest.raises(B.CeError) as ex:
        B.ce_backward_noalloc(p, fake, 0, fake, 0)
    assert ex.value.status == B.CE_ERR_ARG
    B.ce_plan_destroy(p)


@pytest.mark.parametrize("frac", [0.0, 0.3, 0.7, 1.0])
@pytest.mark.parametrize("name", ["C1", "C2s", "C3s", "C4s", "C5bs"])
def test_checkpoint_choice_matches_oracle(name, frac):
    """ce_plan_create_ex with a save budget keeps the same intermediates as
    the oracle's keep-or-recompute choice (Section 3.3), with the same bytes
    and remaining recompute multiplications; the backward's workspace covers
    the forward's whenever anything is kept."""
    w = W.PARITY_WORKLOADS[name]
    elem = 2 if w.dtype == "bf16" else 4
    e = O.bind(O.parse(w.spec), w.shapes)
    t = O.optimal_tree(e)[0]
    total = O.checkpoint_choice(e, t, 10 ** 18, elem)[1]
    budget = int(frac * total)
    x = B.ce_expr_parse(w.spec, w.shapes)
    p = B.ce_plan_create_ex(x, B.CE_COST_FWD, B.CE_BF16 if elem == 2 else B.CE_F32,
                            B.CE_FLAG_NO_FUSION, save_budget=budget)
    B.ce_expr_destroy(x)
    try:
        mask, nbytes, rec = B.ce_plan_checkpoint(p)
        kept, wb, rest = O.checkpoint_choice(e, t, budget, elem)
        assert mask == sum(1 << s for s in kept)
        assert (nbytes, rec) == (wb, rest)
        if mask:
            assert B.ce_plan_workspace_size(p, 1) >= B.ce_plan_workspace_size(p, 0) >= nbytes
    finally:
        B.ce_plan_destroy(p)


def test_checkpoint_keeps_tensor_train_fusion():
    """Under a save budget that cannot hold the tensor-train producer's
    result, the forward stays fused (that result never reaches memory) and
    only the small merged factors are kept; a budget that holds it unfuses
    the forward and keeps it, so the backward recomputes nothing."""
    w = W.WORKLOADS["C4"]
    x = B.ce_expr_parse(w.spec, w.shapes)
    try:
        p0 = B.ce_plan_create(x, B.CE_COST_FWD, B.CE_F32, 0)
        fused_ws = B.ce_plan_workspace_size(p0, 0)
        big = 4 * 64 * 128 * 2 * 16 * 28 * 28   # the rank-expanded input, fp32
        small = B.ce_plan_create_ex(x, B.CE_COST_FWD, B.CE_F32, 0, save_budget=16 << 20)
        whole = B.ce_plan_create_ex(x, B.CE_COST_FWD, B.CE_F32, 0, save_budget=big + (1 << 20))
    finally:
        B.ce_expr_destroy(x)
    try:
        mask, nbytes, rec = B.ce_plan_checkpoint(small)
        assert "fused tensor-train" in B.ce_plan_describe(small)
        assert 0 < nbytes < (1 << 20) and rec > 0
        assert B.ce_plan_workspace_size(small, 0) < fused_ws + (1 << 20)
        mask, nbytes, rec = B.ce_plan_checkpoint(whole)
        assert "fused tensor-train" not in B.ce_plan_describe(whole)
        assert nbytes >= big and rec == 0
    finally:
        for p in (p0, small, whole):
            B.ce_plan_destroy(p)


@pytest.mark.parametrize("name", ["C2s", "C4s", "C5bs", "rtt_conv", "tr_conv"])
def test_cost_cap_plan_matches_oracle(name):
    """ce_plan_create_ex with a per-step cost cap (Section 3.2, Figure 2)
    returns the oracle's capped tree, or CE_ERR_UNSUPPORTED when the oracle
    finds none."""
    if name in PAPER_SHAPES:
        w = W.Workload(name, STRINGS[name][0], tuple(PAPER_SHAPES[name]), "f32", 0, (), ())
    else:
        w = W.PARITY_WORKLOADS[name]
    e = O.bind(O.parse(w.spec), w.shapes)
    t0 = O.optimal_tree(e)[0]
    steps0 = O.step_costs(e, t0)
    for cap in sorted(set(steps0), reverse=True)[:3] + [max(steps0) - 1, min(steps0)]:
        tree, cost = O.optimal_tree(e, max_step_cost=cap)
        x = B.ce_expr_parse(w.spec, w.shapes)
        try:
            if tree is None:
                with pytest.raises(B.CeError) as ex:
                    B.ce_plan_create_ex(x, B.CE_COST_FWD, B.CE_F32, 0, max_step_cost=cap)
                assert ex.value.status == B.CE_ERR_UNSUPPORTED
                continue
            p = B.ce_plan_create_ex(x, B.CE_COST_FWD, B.CE_F32, 0, max_step_cost=cap)
        finally:
            B.ce_expr_destroy(x)
        try:
            assert _steps(p) == _oracle_steps(e, tree), (name, cap)
            assert B.ce_plan_cost(p)[0] == cost
        finally:
            B.ce_plan_destroy(p)


@pytest.mark.parametrize("name", ["C2", "C4", "C5b"])
def test_max_batch(name):
    """The one-layer analogue of the paper's maximum-batch table (Section 5,
    Table 3) under an 11 GiB budget: the returned batch fits and one more
    does not, and the planned order admits at least the batch of the
    left-to-right order with recomputation, which admits at least that of
    left-to-right keeping every intermediate (both unfused)."""
    import paper_2401_03384_amd as P
    w = W.WORKLOADS[name]
    budget = 11 << 30
    opt = P.max_batch(w.spec, w.shapes, budget, w.dtype)
    ckpt = P.max_batch(w.spec, w.shapes, budget, w.dtype, "ltr", fusion=False)
    keep = P.max_batch(w.spec, w.shapes, budget, w.dtype, "ltr", save=True, fusion=False)
    assert opt >= ckpt >= keep >= 1

    def need(bs, **kw):
        shp = [list(s) for s in w.shapes]
        shp[0][0] = bs
        return P.step_bytes(P.Plan(w.spec, shp, w.dtype, **kw))

    assert need(opt) <= budget < need(opt + 1)
    n = len(w.shapes)
    ltr = [(0, 1)] + [(0, n - 1 - k) for k in range(1, n - 1)]
    assert need(keep, path=ltr, flags=B.CE_FLAG_SAVE_INTERMEDIATES | B.CE_FLAG_NO_FUSION) <= budget
    assert need(keep + 1, path=ltr, flags=B.CE_FLAG_SAVE_INTERMEDIATES | B.CE_FLAG_NO_FUSION) > budget


def _plan_strided(spec, shapes, strides, mode=B.CE_COST_FWD, path=None):
    e = B.ce_expr_parse(spec, shapes)
    try:
        for l, s in strides.items():
            B.ce_expr_set_stride(e, l, s)
        if path is not None:
            return B.ce_plan_create_with_path(e, path, B.CE_F32, 0)
        return B.ce_plan_create(e, mode, B.CE_F32, 0)
    finally:
        B.ce_expr_destroy(e)


@pytest.mark.parametrize("scale", [1, 8])
@pytest.mark.parametrize("name", [r[0] for r in W.RESNET34_CONVS])
def test_strided_planner_matches_oracle(name, scale):
    """ResNet-34 convolutions as CP layers (strides 1 and 2, 7x7, 3x3, 1x1),
    full and reduced size: the planner's tree, per-step multiplications and
    totals equal the oracle's in both cost modes, the left-to-right cost too,
    and the output shape is ceil(size / stride)."""
    w, st = W.resnet34_cp_layer(name, batch=128 if scale == 1 else 2, scale=scale)
    e = O.bind(O.parse(w.spec), w.shapes, strides=st)
    for mode, cmode in (("fwd", B.CE_COST_FWD), ("train_paper", B.CE_COST_TRAIN_PAPER)):
        tree, cost = O.optimal_tree(e, mode)
        p = _plan_strided(w.spec, w.shapes, st, cmode)
        try:
            assert _steps(p) == _oracle_steps(e, tree), (name, mode)
            total, fwd = B.ce_plan_cost(p)
            assert total == cost and fwd == O.tree_cost(e, tree, "fwd")
            assert B.ce_plan_left_to_right_cost(p) == O.tree_cost(e, O.left_to_right_tree(5), mode)
        finally:
            B.ce_plan_destroy(p)
    x = B.ce_expr_parse(w.spec, w.shapes)
    for l, s in st.items():
        B.ce_expr_set_stride(x, l, s)
    assert B.ce_expr_output_shape(x) == tuple(w.out_shape)
    B.ce_expr_destroy(x)


def test_stride_errors():
    x = B.ce_expr_parse("bshw,tshw->bthw|hw", [(1, 2, 5, 5), (3, 2, 3, 3)])
    try:
        for label, s, status in (("h", 0, B.CE_ERR_ARG), ("q", 2, B.CE_ERR_ARG),
                                 ("s", 2, B.CE_ERR_ARG)):
            with pytest.raises(B.CeError) as ex:
                B.ce_expr_set_stride(x, label, s)
            assert ex.value.status == status
    finally:
        B.ce_expr_destroy(x)
    x = B.ce_expr_parse("bfshw,fghw,sthw->bgthw|hw", [(1, 2, 2, 7, 7), (2, 2, 3, 3), (2, 2, 3, 3)])
    with pytest.raises(B.CeError) as ex:
        B.ce_expr_set_stride(x, "h", 2)
    assert ex.value.status == B.CE_ERR_UNSUPPORTED
    B.ce_expr_destroy(x)


@pytest.mark.parametrize("name", ["C4", "C4s", "C4w", "C4x2", "C4x4", "C4x1"])
def test_tensor_train_forward_fused(name):
    """The reshaped tensor-train layer's contraction X x W12 and the
    convolution consuming its result run as one fused launch: the forward
    workspace holds only the two merged cores (no X12)."""
    w = W.WORKLOADS.get(name) or W.PARITY_WORKLOADS[name]
    p = _plan(w.spec, w.shapes)
    try:
        text = B.ce_plan_describe(p)
        fwd = [l for l in text.splitlines() if l.startswith("  fwd ")]
        assert sum("tt_fwd<" in l for l in fwd) == 1 and sum("tt_prep" in l for l in fwd) == 1, text
        assert len(fwd) == 4, text
        e = O.bind(O.parse(w.spec), w.shapes)
        tree = O.optimal_tree(e)[0]
        x12 = max(O.intermediate_size(e, O.leaves(a) + O.leaves(b)) for a, b in O.post_order_steps(tree)[:-1])
        assert B.ce_plan_workspace_size(p, 0) < x12 * 4
    finally:
        B.ce_plan_destroy(p)
