"""Pins for the oracle's evaluators (CPU): the plain definition, every
pairwise tree, the dense reconstruction, closed forms and library routines
(PyTorch CPU float64 convolutions, numpy.einsum)."""
import itertools

import numpy as np
import pytest
import torch

import oracle as O
from conftest import load_layer_strings

STRINGS = load_layer_strings()
rng = np.random.default_rng(1234)


def _e(spec, shapes, **kw):
    return O.bind(O.parse(spec), shapes, **kw)


def _rand(shapes, seed=0):
    g = np.random.default_rng(seed)
    return [g.standard_normal(s) for s in shapes]


TINY = {
    "cp_conv": [(2, 3, 5, 4), (2, 2), (2, 3), (2, 3), (2, 3)],
    "tucker_conv": [(2, 3, 4, 5), (2, 2), (2, 3), (2, 2, 3, 2)],
    "tt_conv": [(1, 3, 5, 4), (2, 2), (2, 2, 3), (2, 2, 2), (2, 3)],
    "tr_conv": [(1, 2, 4, 4), (2, 2, 2), (2, 2, 3), (2, 2, 3), (2, 2, 2)],
    "rcp_conv": [(1, 2, 1, 2, 4, 3), (2, 2, 2), (2, 1, 1), (2, 2, 2), (2, 3, 2)],
    "rtt_conv": [(1, 2, 1, 2, 4, 3), (2, 2, 2), (2, 2, 1, 1), (2, 2, 2, 2), (2, 3, 2)],
    "standard_conv": [(2, 3, 5, 4), (2, 3, 3, 2)],
    "separable_depthwise": [(2, 3, 5, 4), (3, 3), (3, 2)],
}


@pytest.mark.parametrize("name", sorted(TINY))
def test_definition_equals_every_pairwise_tree(name):
    spec = STRINGS[name][0]
    shapes = TINY[name]
    e = _e(spec, shapes)
    arr = _rand(shapes, seed=len(name))
    y = O.eval_definition(e, arr)
    n_trees = 0
    for t in O.all_trees(range(e.n)):
        yp = O.eval_pairwise(e, arr, t)
        np.testing.assert_allclose(yp, y, rtol=1e-12, atol=1e-12 * np.abs(y).max())
        n_trees += 1
    assert n_trees == O.count_trees(e.n)


@pytest.mark.parametrize("name", ["cp_conv", "tucker_conv", "rcp_conv", "rtt_conv", "standard_conv"])
def test_dense_equals_definition(name):
    spec = STRINGS[name][0]
    e = _e(spec, TINY[name])
    arr = _rand(TINY[name], seed=7)
    np.testing.assert_allclose(O.eval_dense(e, arr), O.eval_definition(e, arr), rtol=1e-12,
                               atol=1e-12)


@pytest.mark.parametrize("K,L", [(3, 3), (5, 3), (2, 4), (1, 3), (4, 1)])
def test_standard_conv_matches_torch_conv2d(K, L):
    """bshw,tshw->bthw|hw is the standard 2-D convolution layer (Section 2.3);
    PyTorch's conv2d(padding='same') is cross-correlation with
    floor((K-1)/2) zeros before."""
    X = rng.standard_normal((2, 3, 9, 7))
    W = rng.standard_normal((4, 3, K, L))
    e = _e("bshw,tshw->bthw|hw", [X.shape, W.shape])
    ref = torch.nn.functional.conv2d(torch.tensor(X), torch.tensor(W), padding="same").numpy()
    np.testing.assert_allclose(O.eval_pairwise(e, [X, W], (0, 1)), ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(O.eval_dense(e, [X, W]), ref, rtol=1e-12, atol=1e-12)


def test_conv1d_and_group_conv1d_match_torch():
    X = rng.standard_normal((2, 3, 11))
    W = rng.standard_normal((4, 3, 3))
    e = _e("bsh,tsh->bth|h", [X.shape, W.shape])
    ref = torch.nn.functional.conv1d(torch.tensor(X), torch.tensor(W), padding="same").numpy()
    np.testing.assert_allclose(O.eval_pairwise(e, [X, W], (0, 1)), ref, rtol=1e-12, atol=1e-12)
    # grouped: gtsh,bgsh->bgth|h (Section 3.1); the input is the larger-h operand
    G, T, S = 2, 3, 2
    Wg = rng.standard_normal((G, T, S, 3))
    Xg = rng.standard_normal((2, G, S, 10))
    e = _e("gtsh,bgsh->bgth|h", [Wg.shape, Xg.shape])
    assert e.feature == {"h": 1}
    ref = torch.nn.functional.conv1d(torch.tensor(Xg.reshape(2, G * S, 10)),
                                     torch.tensor(Wg.reshape(G * T, S, 3)), padding="same",
                                     groups=G).numpy().reshape(2, G, T, 10)
    np.testing.assert_allclose(O.eval_pairwise(e, [Wg, Xg], (0, 1)), ref, rtol=1e-12, atol=1e-12)


def test_separable_depthwise_matches_torch_grouped_conv2d():
    S = 4
    X = rng.standard_normal((2, S, 8, 6))
    kh = rng.standard_normal((S, 3))
    kw = rng.standard_normal((S, 5))
    e = _e("bshw,sh,sw->bshw|hw", [X.shape, kh.shape, kw.shape])
    w = np.einsum("sh,sw->shw", kh, kw)[:, None]
    ref = torch.nn.functional.conv2d(torch.tensor(X), torch.tensor(w), padding="same",
                                     groups=S).numpy()
    for t in O.all_trees(range(3)):
        np.testing.assert_allclose(O.eval_pairwise(e, [X, kh, kw], t), ref, rtol=1e-12,
                                   atol=1e-12)


def test_tucker_with_identity_factors_is_standard_conv():
    S, T = 3, 4
    X = rng.standard_normal((2, S, 7, 6))
    G = rng.standard_normal((S, T, 3, 3))
    e = _e("bshw,sp,pqhw,qt->bthw|hw", [X.shape, (S, S), G.shape, (T, T)])
    y = O.eval_pairwise(e, [X, np.eye(S), G, np.eye(T)], O.optimal_tree(e)[0])
    ref = torch.nn.functional.conv2d(torch.tensor(X), torch.tensor(G.transpose(1, 0, 2, 3)),
                                     padding="same").numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_unit_filters_reduce_to_plain_einsum():
    shapes = [(2, 3, 5, 4), (2, 3), (2, 4), (2, 1), (2, 1)]
    e = _e("bshw,rs,rt,rh,rw->bthw|hw", shapes)
    X, Us, Ut, Kh, Kw = _rand(shapes, seed=3)
    ref = np.einsum("bshw,rs,rt,r,r->bthw", X, Us, Ut, Kh[:, 0], Kw[:, 0], optimize=False)
    for t in O.all_trees(range(5)):
        np.testing.assert_allclose(O.eval_pairwise(e, [X, Us, Ut, Kh, Kw], t), ref, rtol=1e-12,
                                   atol=1e-12)


@pytest.mark.parametrize("K", [3, 5, 4])
def test_rank1_impulse_closed_form(K):
    """R = 1, X = e_{b0,s0,h0,w0}:
    Y[b,t,h,w] = d(b,b0) U_t[0,t] U_s[0,s0] K_h[0,h0-h+c] K_w[0,w0-w+c]."""
    B, S, T, H, W = 2, 3, 2, 7, 6
    c = (K - 1) // 2
    Us, Ut = rng.standard_normal((1, S)), rng.standard_normal((1, T))
    Kh, Kw = rng.standard_normal((1, K)), rng.standard_normal((1, K))
    e = _e("bshw,rs,rt,rh,rw->bthw|hw", [(B, S, H, W), Us.shape, Ut.shape, Kh.shape, Kw.shape])
    for b0, s0, h0, w0 in [(1, 2, 3, 2), (0, 0, 0, 5), (1, 1, 6, 0)]:
        X = np.zeros((B, S, H, W))
        X[b0, s0, h0, w0] = 1.0
        y = O.eval_pairwise(e, [X, Us, Ut, Kh, Kw], O.optimal_tree(e)[0])
        ref = np.zeros_like(y)
        for t, h, w in itertools.product(range(T), range(H), range(W)):
            kh, kw = h0 - h + c, w0 - w + c
            if 0 <= kh < K and 0 <= kw < K:
                ref[b0, t, h, w] = Ut[0, t] * Us[0, s0] * Kh[0, kh] * Kw[0, kw]
        np.testing.assert_allclose(y, ref, rtol=1e-13, atol=1e-15)


def test_constant_input_border_closed_form():
    """R = 1, X = 1: interior entries are U_t[0,t] sum(U_s) sum(K_h) sum(K_w);
    border rows and columns drop the taps that fall outside."""
    B, S, T, H, W, K = 1, 3, 2, 6, 5, 3
    Us, Ut = rng.standard_normal((1, S)), rng.standard_normal((1, T))
    Kh, Kw = rng.standard_normal((1, K)), rng.standard_normal((1, K))
    e = _e("bshw,rs,rt,rh,rw->bthw|hw", [(B, S, H, W), Us.shape, Ut.shape, Kh.shape, Kw.shape])
    y = O.eval_dense(e, [np.ones((B, S, H, W)), Us, Ut, Kh, Kw])
    c = 1
    for h, w in itertools.product(range(H), range(W)):
        sh = sum(Kh[0, k] for k in range(K) if 0 <= h + k - c < H)
        sw = sum(Kw[0, k] for k in range(K) if 0 <= w + k - c < W)
        np.testing.assert_allclose(y[0, :, h, w], Ut[0] * Us.sum() * sh * sw, rtol=1e-13)


def _circ_fft(arrays_axes, N):
    """Circular convolution of 1-D signals (zero-padded to N) by the DFT
    identity: ifft(prod fft(a_k, N))."""
    f = np.ones(N, dtype=complex)
    for a in arrays_axes:
        f = f * np.fft.fft(a, N)
    return np.fft.ifft(f).real


@pytest.mark.parametrize("sizes", [(9, 3, 4), (6, 6, 6), (5, 7, 2), (4, 4, 9)])
def test_multiway_circular_matches_dft(sizes):
    """A label held by three operands is convolved circularly (Appendix B):
    the definition and every pairwise tree equal the DFT identity (numpy.fft)
    with N the largest size; the result is the same in every order
    (commutative and associative)."""
    g = np.random.default_rng(sum(sizes))
    arr = [g.standard_normal(n) for n in sizes]
    e = _e("i,i,i->i|i", [(n,) for n in sizes])
    assert e.circular == {"i"} and e.out_sizes["i"] == max(sizes)
    ref = _circ_fft(arr, max(sizes))
    np.testing.assert_allclose(O.eval_definition(e, arr), ref, rtol=1e-12, atol=1e-12)
    for t in O.all_trees(range(3)):
        np.testing.assert_allclose(O.eval_pairwise(e, arr, t), ref, rtol=1e-12, atol=1e-12)


def test_two_way_circular_matches_dft():
    """A two-way label chosen circular: batched 1-D circular convolution,
    y[b, t] = sum_s x[b, s] (*) f[t, s], by the DFT along h."""
    g = np.random.default_rng(3)
    X, F = g.standard_normal((2, 3, 8)), g.standard_normal((4, 3, 5))
    e = O.bind(O.parse("bsh,tsh->bth|h"), [X.shape, F.shape], circular=("h",))
    ref = np.fft.ifft(np.einsum("bsh,tsh->bth", np.fft.fft(X, 8, axis=-1),
                                np.fft.fft(F, 8, axis=-1))).real
    np.testing.assert_allclose(O.eval_definition(e, [X, F]), ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(O.eval_pairwise(e, [X, F], (0, 1)), ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("name", ["interleaved_group", "interleaved_group_sec2"])
def test_interleaved_group_conv_matches_dft(name):
    """The interleaved group convolutions of Section 2.2 and Appendix A.3.1
    (h, w held by three operands, circular): the definition and every tree
    equal the 2-D DFT identity, a product of the three transforms summed over
    the contracted channels."""
    spec = STRINGS[name][0]
    shapes = [(1, 2, 2, 5, 6), (2, 2, 3, 3), (3, 2, 2, 4)] if name == "interleaved_group" \
        else [(1, 2, 2, 5, 6), (2, 2, 3, 3), (2, 3, 2, 4)]
    g = np.random.default_rng(4)
    arr = [g.standard_normal(s) for s in shapes]
    e = _e(spec, shapes)
    N = (5, 6)
    F = [np.fft.fft2(a, N) for a in arr]
    lhs, out = spec.split("|")[0].split("->")
    ops = lhs.split(",")
    ref = np.fft.ifft2(np.einsum(",".join(ops) + "->" + out, *F), axes=(-2, -1)).real
    np.testing.assert_allclose(O.eval_definition(e, arr), ref, rtol=1e-11, atol=1e-11)
    for t in O.all_trees(range(3)):
        np.testing.assert_allclose(O.eval_pairwise(e, arr, t), ref, rtol=1e-11, atol=1e-11)


def test_circular_cost_hand_values():
    """A circular step meets every pair of positions once: sizes 9, 3, 4 give
    9*3 then (N = 9)*4 along ((0,1),2), and 3*4 then 9*9 along (0,(1,2))
    (merging two holders gives an N-position tensor)."""
    e = _e("i,i,i->i|i", [(9,), (3,), (4,)])
    assert O.step_costs(e, ((0, 1), 2)) == [27, 36]
    assert O.step_costs(e, (0, (1, 2))) == [12, 81]
    assert O.intermediate_size(e, (1, 2)) == 9
    assert O.optimal_tree(e) == (((0, 1), 2), 63)


def test_self_contracted_label_is_presummed():
    X = rng.standard_normal((2, 3, 4))
    A = rng.standard_normal((4, 5))
    e = _e("bsm,mt->bt", [X.shape, A.shape])   # s is self-contracted
    ref = np.einsum("bsm,mt->bt", X, A)
    np.testing.assert_allclose(O.eval_pairwise(e, [X, A], (0, 1)), ref, rtol=1e-12)
    np.testing.assert_allclose(O.eval_definition(e, [X, A]), ref, rtol=1e-12)


STRIDED = [
    # (H, W, K, stride): odd and even feature sizes, 3x3, 7x7 (a ResNet stem),
    # 1x1 (a strided shortcut), strides 2 and 3
    (9, 9, 3, 2), (8, 10, 3, 2), (11, 12, 7, 2), (8, 7, 1, 2), (10, 9, 3, 3),
]


@pytest.mark.parametrize("H,W_,K,s", STRIDED)
def test_strided_conv_matches_torch(H, W_, K, s):
    """A strided convolution (Appendix B, a non-commutative variety) against
    PyTorch CPU float64 conv2d(stride=s, padding=(K-1)//2) and its autograd:
    the definition, the pairwise evaluation and the dense evaluation."""
    g = np.random.default_rng(40 + K + s)
    X = g.standard_normal((2, 3, H, W_))
    F = g.standard_normal((4, 3, K, K))
    e = O.bind(O.parse("bshw,tshw->bthw|hw"), [X.shape, F.shape], strides={"h": s, "w": s})
    xt = torch.tensor(X, requires_grad=True)
    ft = torch.tensor(F, requires_grad=True)
    y = torch.nn.functional.conv2d(xt, ft, stride=s, padding=(K - 1) // 2)
    assert tuple(e.out_sizes[l] for l in "bthw") == tuple(y.shape)
    dy = g.standard_normal(tuple(y.shape))
    (y * torch.tensor(dy)).sum().backward()
    ref = y.detach().numpy()
    t = O.optimal_tree(e)[0]
    np.testing.assert_allclose(O.eval_definition(e, [X, F]), ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(O.eval_pairwise(e, [X, F], t), ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(O.eval_dense(e, [X, F]), ref, rtol=1e-12, atol=1e-12)
    for gp, gd, tt in zip(O.grads_pairwise(e, [X, F], t, dy), O.grads_dense(e, [X, F], dy),
                          (xt, ft)):
        np.testing.assert_allclose(gp, tt.grad.numpy(), rtol=1e-11, atol=1e-11)
        np.testing.assert_allclose(gd, tt.grad.numpy(), rtol=1e-11, atol=1e-11)


def test_strided_cp_layer_every_tree_matches_torch():
    """CP layer with stride 2 on h and w: every one of the 105 trees, the
    definition and the dense evaluation equal torch conv2d with the
    reconstructed kernel; the convolved labels of every intermediate holding
    both sides have ceil(I / 2) positions."""
    g = np.random.default_rng(41)
    B, S, T, R, H, W_, K = 2, 3, 4, 2, 7, 8, 3
    arr = [g.standard_normal(s) for s in [(B, S, H, W_), (R, S), (R, T), (R, K), (R, K)]]
    e = O.bind(O.parse("bshw,rs,rt,rh,rw->bthw|hw"), [a.shape for a in arr],
               strides={"h": 2, "w": 2})
    Wd = np.einsum("rs,rt,rh,rw->tshw", *arr[1:])
    ref = torch.nn.functional.conv2d(torch.tensor(arr[0]), torch.tensor(Wd), stride=2,
                                     padding=1).numpy()
    np.testing.assert_allclose(O.eval_definition(e, arr), ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(O.eval_dense(e, arr), ref, rtol=1e-12, atol=1e-12)
    for t in O.all_trees(range(5)):
        np.testing.assert_allclose(O.eval_pairwise(e, arr, t), ref, rtol=1e-11, atol=1e-11)
    assert O.intermediate_size(e, (0, 3)) == B * S * R * 4 * W_      # h convolved: ceil(7/2)
    assert O.intermediate_size(e, (0, 1, 3, 4)) == B * R * 4 * 4


def test_strided_cost():
    """The strided step counts output positions times taps: a 3x3 stride-2
    convolution of X[2, 3, 9, 9] with W[4, 3, 3, 3] does 2*4*3*5*5*3*3
    multiplications; with stride 1 it would be 2*4*3*9*9*3*3."""
    e = O.bind(O.parse("bshw,tshw->bthw|hw"), [(2, 3, 9, 9), (4, 3, 3, 3)],
               strides={"h": 2, "w": 2})
    assert O.step_cost(e, (0,), (1,)) == 2 * 4 * 3 * 5 * 5 * 3 * 3
    # training (Appendix B): g1 = output * filter, g2 = feature * output per label
    assert O.step_cost(e, (0,), (1,), "train_paper") == 2 * 4 * 3 * (
        (5 * 3) ** 2 + (5 * 3) ** 2 + (9 * 5) ** 2)
    e1 = O.bind(O.parse("bshw,tshw->bthw|hw"), [(2, 3, 9, 9), (4, 3, 3, 3)])
    assert O.step_cost(e1, (0,), (1,)) == 2 * 4 * 3 * 9 * 9 * 3 * 3
