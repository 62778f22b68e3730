"""Float64 gradients of a conv_einsum layer (test infrastructure).

grads_pairwise  reverse pass along a tree.  For every step T = f(T1, T2) it
                forms dL/dT1 = g1(dL/dT, T2) and dL/dT2 = g2(T1, dL/dT)
                (Appendix B, 'Modification of the cost model for training');
                intermediates of the forward pass are recomputed first, as
                gradient checkpointing does (Section 3.3).  Each g is the
                adjoint of the step written tap by tap: the feature side
                receives the shifted-back einsum of dT with the filter tap,
                the filter tap receives the einsum of the shifted feature
                with dT.
grads_dense     chain rule through the reconstructed dense kernel W:
                dX is the transposed convolution of dY with W,
                dW[.., k] = sum over batch and positions of X[p + k - c] dY[p],
                and each factor's gradient is the einsum of dW with all other
                factors (W is a plain einsum of the factors).
"""
from __future__ import annotations

import itertools

import numpy as np

from .cost import kept_labels, label_size, stride_of
from .evaluate import (_letters, _einsum, shift, shift_adjoint, step_convs, circ_shift,
                       circ_shift_adjoint,
                       leaf_tensor, dense_kernel, pair_step)
from .notation import Expr


def pair_adjoint(expr, letters, a, A, b, B, dc):
    """Gradients of one pairwise step with respect to its two inputs."""
    la, lb = kept_labels(expr, A), kept_labels(expr, B)
    lc = kept_labels(expr, tuple(A) + tuple(B))
    convs = step_convs(expr, A, B)
    taps = []
    for l, fa in convs:
        taps.append(range(label_size(expr, B, l) if fa or fa is None else label_size(expr, A, l)))
    da = np.zeros_like(a)
    db = np.zeros_like(b)
    for combo in itertools.product(*taps):
        xa, xb, ca, cb = a, b, list(la), list(lb)
        a_shifts, b_shifts, a_taps, b_taps, a_circ = [], [], [], [], []
        for (l, fa), k in zip(convs, combo):
            s = stride_of(expr, l)
            if fa is None:
                N = label_size(expr, tuple(A) + tuple(B), l)
                a_circ.append((l, k, N, xa.shape[ca.index(l)]))
                xa = circ_shift(xa, ca.index(l), k, N)
                b_taps.append((l, k))
                xb = np.take(xb, k, axis=cb.index(l))
                cb.remove(l)
            elif fa:
                K = label_size(expr, B, l)
                a_shifts.append((l, k, K, xa.shape[ca.index(l)], s))
                xa = shift(xa, ca.index(l), k, K, s)
                b_taps.append((l, k))
                xb = np.take(xb, k, axis=cb.index(l))
                cb.remove(l)
            else:
                K = label_size(expr, A, l)
                b_shifts.append((l, k, K, xb.shape[cb.index(l)], s))
                xb = shift(xb, cb.index(l), k, K, s)
                a_taps.append((l, k))
                xa = np.take(xa, k, axis=ca.index(l))
                ca.remove(l)
        # adjoint w.r.t. the (shifted / tap-sliced) view of a
        ga = _einsum(letters, dc, lc, xb, cb, ca)
        for l, k, K, n, s in a_shifts:
            ga = shift_adjoint(ga, ca.index(l), k, K, n, s)
        for l, k, N, n in a_circ:
            ga = circ_shift_adjoint(ga, ca.index(l), k, N, n)
        idx = [slice(None)] * da.ndim
        for l, k in a_taps:
            idx[la.index(l)] = k
        if a_taps:
            # ca lacks the tapped labels: place the slice at its tap
            da[tuple(idx)] += ga
        else:
            da += ga
        gb = _einsum(letters, xa, ca, dc, lc, cb)
        for l, k, K, n, s in b_shifts:
            gb = shift_adjoint(gb, cb.index(l), k, K, n, s)
        idx = [slice(None)] * db.ndim
        for l, k in b_taps:
            idx[lb.index(l)] = k
        if b_taps:
            db[tuple(idx)] += gb
        else:
            db += gb
    return da, db


def grads_pairwise(expr: Expr, arrays, tree, dy):
    """[dL/d operand_i] for L = <Y, dy>, along `tree`."""
    letters = _letters(expr)
    vals = {}

    def fwd(t):
        if isinstance(t, int):
            a, _ = leaf_tensor(expr, arrays, t)
            vals[(t,)] = a
            return a, (t,)
        a, A = fwd(t[0])
        b, B = fwd(t[1])
        c, _ = pair_step(expr, letters, a, A, b, B)
        vals[A + B] = c
        return c, A + B

    # a single operand (no pairwise step): its gradient is dy broadcast over
    # the labels its pre-sum removed
    _, S = fwd(tree)
    lroot = kept_labels(expr, S)
    droot = np.transpose(np.asarray(dy, np.float64), [expr.output.index(l) for l in lroot])
    grads = {}

    def bwd(t, dt):
        if isinstance(t, int):
            grads[t] = dt
            return
        A = tuple(_leaves(t[0]))
        B = tuple(_leaves(t[1]))
        a, b = vals[A], vals[B]
        da, db = pair_adjoint(expr, letters, a, A, b, B, dt)
        bwd(t[0], da)
        bwd(t[1], db)

    bwd(tree, droot)
    out = []
    for i in range(expr.n):
        g = grads[i]                      # kept-label order
        li = list(expr.inputs[i])
        keep = kept_labels(expr, (i,))
        rest = [l for l in li if l in keep]
        g = np.transpose(g, [keep.index(l) for l in rest])
        # undo the pre-sum of self-contracted labels: broadcast
        gi = g.reshape([expr.sizes[i][l] if l in keep else 1 for l in li])
        out.append(np.broadcast_to(gi, [expr.sizes[i][l] for l in li]).copy())
    return out


def _leaves(t):
    return (t,) if isinstance(t, int) else _leaves(t[0]) + _leaves(t[1])


def grads_dense(expr: Expr, arrays, dy, feature_operand: int = 0):
    """[dL/d operand_i] via the reconstructed dense kernel."""
    W, lw = dense_kernel(expr, arrays, feature_operand)
    X = np.asarray(arrays[feature_operand], np.float64)
    lx = list(expr.inputs[feature_operand])
    if kept_labels(expr, (feature_operand,)) != [l for l in lx]:
        raise NotImplementedError("feature operand with self-contracted labels")
    dy = np.asarray(dy, np.float64)
    letters = _letters(expr)
    convs = list(expr.conv)
    Ks = [W.shape[lw.index(l)] for l in convs]
    lw_red = [l for l in lw if l not in convs]
    # Output position p read the zero-padded X at s*p + k for tap k (padding c
    # before, K-1-c after): dX is accumulated in the padded frame at those
    # positions and cropped; dW[k] pairs the same window of X with dY.
    pads_x = [(0, 0)] * X.ndim
    for l, K in zip(convs, Ks):
        c = (K - 1) // 2
        pads_x[lx.index(l)] = (c, K - 1 - c)
    Xp = np.pad(X, pads_x)
    dXp = np.zeros_like(Xp)
    dW = np.zeros_like(W)
    for combo in itertools.product(*[range(K) for K in Ks]):
        xwin = [slice(None)] * X.ndim
        widx = [slice(None)] * W.ndim
        for l, K, k in zip(convs, Ks, combo):
            s = stride_of(expr, l)
            m = dy.shape[expr.output.index(l)]
            xwin[lx.index(l)] = slice(k, k + s * (m - 1) + 1, s)
            widx[lw.index(l)] = k
        Wk = W[tuple(widx)]
        dXp[tuple(xwin)] += _einsum(letters, dy, expr.output, Wk, lw_red, lx)
        dW[tuple(widx)] += _einsum(letters, Xp[tuple(xwin)], lx, dy, expr.output, lw_red)
    crop = [slice(None)] * X.ndim
    for l, K in zip(convs, Ks):
        c = (K - 1) // 2
        crop[lx.index(l)] = slice(c, c + X.shape[lx.index(l)])
    dX = dXp[tuple(crop)]
    out = []
    for i in range(expr.n):
        if i == feature_operand:
            out.append(dX)
            continue
        others = [j for j in range(expr.n) if j not in (i, feature_operand)]
        li = list(expr.inputs[i])
        for l in li:
            if l not in lw and not any(l in expr.inputs[j] for j in others):
                raise NotImplementedError("factor with a self-contracted label")
        sub = ",".join(["".join(letters[l] for l in lw)] +
                       ["".join(letters[l] for l in expr.inputs[j]) for j in others]) + \
            "->" + "".join(letters[l] for l in li)
        ops = [dW] + [np.asarray(arrays[j], np.float64) for j in others]
        out.append(np.einsum(sub, *ops, optimize=True))
    return out
