"""Pins for the oracle's gradients (CPU): central finite differences,
PyTorch CPU float64 autograd of the dense layer, agreement of every tree, and
the multilinearity identity <T_i, dL/dT_i> = <Y, dY> for every operand."""
import numpy as np
import pytest
import torch

import oracle as O
from conftest import load_layer_strings

STRINGS = load_layer_strings()

CASES = {
    "cp_conv": [(2, 3, 5, 4), (2, 2), (2, 3), (2, 3), (2, 3)],
    "tucker_conv": [(2, 3, 4, 5), (2, 2), (2, 3), (2, 2, 3, 3)],
    "rtt_conv": [(1, 2, 1, 2, 4, 3), (2, 2, 2), (2, 2, 1, 1), (2, 2, 2, 2), (2, 3, 2)],
    "rcp_conv": [(2, 2, 1, 2, 4, 3), (2, 2, 2), (2, 1, 1), (2, 2, 2), (2, 3, 2)],
    "tt_conv": [(1, 3, 5, 4), (2, 2), (2, 2, 3), (2, 2, 2), (2, 3)],
}


def _setup(name, seed=0):
    shapes = CASES[name]
    e = O.bind(O.parse(STRINGS[name][0]), shapes)
    g = np.random.default_rng(seed)
    arr = [g.standard_normal(s) for s in shapes]
    y = O.eval_definition(e, arr)
    dy = g.standard_normal(y.shape)
    return e, arr, y, dy


@pytest.mark.parametrize("name", sorted(CASES))
def test_finite_differences(name):
    e, arr, y, dy = _setup(name)
    t = O.optimal_tree(e)[0]
    grads = O.grads_pairwise(e, arr, t, dy)
    g = np.random.default_rng(5)
    eps = 1e-6
    for i, a in enumerate(arr):
        for _ in range(6):
            idx = tuple(int(g.integers(0, d)) for d in a.shape)
            ap = [x.copy() for x in arr]
            am = [x.copy() for x in arr]
            ap[i][idx] += eps
            am[i][idx] -= eps
            fd = ((O.eval_definition(e, ap) - O.eval_definition(e, am)) * dy).sum() / (2 * eps)
            assert abs(fd - grads[i][idx]) <= 1e-7 * max(1.0, abs(fd)), (i, idx)


@pytest.mark.parametrize("name", ["cp_conv", "tucker_conv", "rtt_conv", "rcp_conv"])
def test_every_tree_gives_the_dense_gradient(name):
    e, arr, y, dy = _setup(name, seed=1)
    ref = O.grads_dense(e, arr, dy)
    for t in O.all_trees(range(e.n)):
        for a, b in zip(O.grads_pairwise(e, arr, t, dy), ref):
            np.testing.assert_allclose(a, b, rtol=1e-11, atol=1e-11 * max(1.0, np.abs(b).max()))


@pytest.mark.parametrize("name", sorted(CASES))
def test_multilinearity_identity(name):
    """Y is linear in each operand, so <T_i, dL/dT_i> = <Y, dY> for every i."""
    e, arr, y, dy = _setup(name, seed=2)
    ydy = float((y * dy).sum())
    for a, g in zip(arr, O.grads_pairwise(e, arr, O.optimal_tree(e)[0], dy)):
        assert abs(float((a * g).sum()) - ydy) <= 1e-11 * max(1.0, abs(ydy))


def test_cp_gradients_match_torch_autograd():
    """Independent library: the CP kernel built with torch.einsum, the layer
    with torch conv2d(padding='same'), gradients by torch autograd."""
    B, S, T, R, H, W, K = 2, 4, 3, 3, 9, 8, 3
    g = np.random.default_rng(9)
    X, Us, Ut, Kh, Kw = [g.standard_normal(s) for s in
                         [(B, S, H, W), (R, S), (R, T), (R, K), (R, K)]]
    dy = g.standard_normal((B, T, H, W))
    e = O.bind(O.parse("bshw,rs,rt,rh,rw->bthw|hw"), [X.shape, Us.shape, Ut.shape, Kh.shape,
                                                      Kw.shape])
    tt = [torch.tensor(a, requires_grad=True) for a in (X, Us, Ut, Kh, Kw)]
    Wd = torch.einsum("rs,rt,rh,rw->tshw", tt[1], tt[2], tt[3], tt[4])
    y = torch.nn.functional.conv2d(tt[0], Wd, padding="same")
    (y * torch.tensor(dy)).sum().backward()
    ours = O.grads_pairwise(e, [X, Us, Ut, Kh, Kw], O.optimal_tree(e)[0], dy)
    np.testing.assert_allclose(O.eval_pairwise(e, [X, Us, Ut, Kh, Kw], O.optimal_tree(e)[0]),
                               y.detach().numpy(), rtol=1e-12, atol=1e-12)
    for a, t in zip(ours, tt):
        np.testing.assert_allclose(a, t.grad.numpy(), rtol=1e-11, atol=1e-11)


def test_tucker_gradients_match_torch_autograd():
    B, S, T, P, Q, H, W, K = 2, 5, 4, 3, 2, 7, 6, 3
    g = np.random.default_rng(10)
    X, Ui, G, Uo = [g.standard_normal(s) for s in [(B, S, H, W), (S, P), (P, Q, K, K), (Q, T)]]
    dy = g.standard_normal((B, T, H, W))
    e = O.bind(O.parse("bshw,sp,pqhw,qt->bthw|hw"), [X.shape, Ui.shape, G.shape, Uo.shape])
    tt = [torch.tensor(a, requires_grad=True) for a in (X, Ui, G, Uo)]
    Wd = torch.einsum("sp,pqhw,qt->tshw", tt[1], tt[2], tt[3])
    y = torch.nn.functional.conv2d(tt[0], Wd, padding="same")
    (y * torch.tensor(dy)).sum().backward()
    ours = O.grads_dense(e, [X, Ui, G, Uo], dy)
    for a, t in zip(ours, tt):
        np.testing.assert_allclose(a, t.grad.numpy(), rtol=1e-11, atol=1e-11)


EDGE = [
    ("ijk->i", [(3, 4, 5)], 0),                 # one operand: a pre-sum only
    ("ijk->kji", [(2, 3, 4)], 0),               # one operand: a transpose
    ("bsm,mt->bt", [(2, 3, 4), (4, 5)], 0),     # s summed away before the step
    ("tsh,bsh->bth|h", [(3, 2, 3), (2, 2, 7)], 0),   # the feature operand second
    ("bsh,tsh->bth|h", [(2, 2, 5), (3, 2, 5)], 1),   # equal sizes, feature operand 1
    ("bshw,tshw->bthw|hw", [(1, 2, 6, 5), (2, 2, 4, 2)], 0),   # even filters
]


@pytest.mark.parametrize("spec,shapes,feat", EDGE, ids=[c[0] for c in EDGE])
def test_finite_differences_edge_cases(spec, shapes, feat):
    """The method's degenerate cases (Section 3.1 case (5) pre-sums, single
    operands, feature side second or chosen on equal sizes, even filters):
    pairwise gradients against central differences of the plain definition."""
    e = O.bind(O.parse(spec), shapes, feature_operand=feat)
    g = np.random.default_rng(11)
    arr = [g.standard_normal(s) for s in shapes]
    y = O.eval_definition(e, arr)
    dy = g.standard_normal(y.shape)
    t = O.optimal_tree(e)[0]
    np.testing.assert_allclose(O.eval_pairwise(e, arr, t), y, rtol=1e-12, atol=1e-12)
    grads = O.grads_pairwise(e, arr, t, dy)
    eps = 1e-6
    for i, a in enumerate(arr):
        for idx in list(np.ndindex(*a.shape))[::max(1, a.size // 12)]:
            ap = [x.copy() for x in arr]
            am = [x.copy() for x in arr]
            ap[i][idx] += eps
            am[i][idx] -= eps
            fd = ((O.eval_definition(e, ap) - O.eval_definition(e, am)) * dy).sum() / (2 * eps)
            assert abs(fd - grads[i][idx]) <= 1e-7 * max(1.0, abs(fd)), (i, idx)


def test_single_operand_gradient_is_a_broadcast():
    """Y[i] = sum_jk X[i,j,k]: dL/dX[i,j,k] = dY[i] for every j, k."""
    e = O.bind(O.parse("ijk->i"), [(3, 4, 5)])
    x = np.random.default_rng(3).standard_normal((3, 4, 5))
    dy = np.array([1.5, -2.0, 0.25])
    (gx,) = O.grads_pairwise(e, [x], 0, dy)
    assert np.array_equal(gx, np.broadcast_to(dy[:, None, None], (3, 4, 5)))


@pytest.mark.parametrize("spec,shapes,strides", [
    ("bshw,rs,rt,rh,rw->bthw|hw", [(1, 2, 5, 6), (2, 2), (2, 3), (2, 3), (2, 3)], {"h": 2, "w": 2}),
    ("bsh,tsh->bth|h", [(2, 2, 9), (3, 2, 4)], {"h": 3}),
    ("tsh,bsh->bth|h", [(3, 2, 1), (2, 2, 7)], {"h": 2}),
])
def test_finite_differences_strided(spec, shapes, strides):
    """Strided convolutions (Appendix B, non-commutative varieties): pairwise
    gradients along the optimal tree against central differences of the
    plain definition."""
    e = O.bind(O.parse(spec), shapes, strides=strides)
    g = np.random.default_rng(12)
    arr = [g.standard_normal(s) for s in shapes]
    y = O.eval_definition(e, arr)
    dy = g.standard_normal(y.shape)
    t = O.optimal_tree(e)[0]
    grads = O.grads_pairwise(e, arr, t, dy)
    eps = 1e-6
    for i, a in enumerate(arr):
        for idx in list(np.ndindex(*a.shape))[::max(1, a.size // 10)]:
            ap = [x.copy() for x in arr]
            am = [x.copy() for x in arr]
            ap[i][idx] += eps
            am[i][idx] -= eps
            fd = ((O.eval_definition(e, ap) - O.eval_definition(e, am)) * dy).sum() / (2 * eps)
            assert abs(fd - grads[i][idx]) <= 1e-7 * max(1.0, abs(fd)), (i, idx)


@pytest.mark.parametrize("spec,shapes,circ", [
    ("i,i,i->i|i", [(9,), (3,), (4,)], ()),
    ("bsh,tsh->bth|h", [(2, 2, 7), (3, 2, 4)], ("h",)),
    ("bmshw,nmhw,tshw->bnthw|hw", [(1, 2, 2, 4, 5), (2, 2, 2, 3), (2, 2, 3, 2)], ()),
])
def test_finite_differences_circular(spec, shapes, circ):
    """Circular (commutative) convolutions, multi-way and two-way: pairwise
    gradients along every tree against central differences of the plain
    definition, and the multilinearity identity."""
    e = O.bind(O.parse(spec), shapes, circular=circ)
    g = np.random.default_rng(13)
    arr = [g.standard_normal(s) for s in shapes]
    y = O.eval_definition(e, arr)
    dy = g.standard_normal(y.shape)
    ydy = float((y * dy).sum())
    for t in O.all_trees(range(e.n)):
        grads = O.grads_pairwise(e, arr, t, dy)
        for a, gr in zip(arr, grads):
            assert abs(float((a * gr).sum()) - ydy) <= 1e-10 * max(1.0, abs(ydy))
    grads = O.grads_pairwise(e, arr, O.optimal_tree(e)[0], dy)
    eps = 1e-6
    for i, a in enumerate(arr):
        for idx in list(np.ndindex(*a.shape))[::max(1, a.size // 10)]:
            ap = [x.copy() for x in arr]
            am = [x.copy() for x in arr]
            ap[i][idx] += eps
            am[i][idx] -= eps
            fd = ((O.eval_definition(e, ap) - O.eval_definition(e, am)) * dy).sum() / (2 * eps)
            assert abs(fd - grads[i][idx]) <= 1e-7 * max(1.0, abs(fd)), (i, idx)
