"""Float64 evaluators of a conv_einsum layer (test infrastructure).

eval_definition  the plain definition, one output entry at a time, written
                 from the primitive definitions of Appendix A (contraction,
                 batch product, outer product, mode-(k,l) convolution) with
                 the same-padding convolution of the reading below.  Pure
                 Python loops: tiny inputs only.
eval_pairwise    the pairwise evaluation along any tree (Section 3.1 atomic
                 operations, Section 3.2 sequencing).  Each step sums the
                 convolved labels' taps explicitly (shift and accumulate) and
                 hands the rest of the step to numpy.einsum.
eval_dense       the reconstructed dense kernel (the factors merged by one
                 einsum, Section 2.3 and Appendix A.3) followed by a direct
                 convolution with the feature operand (zero padding by
                 numpy.pad and shifted slices).

Convolution (reading of Section 2.2 and Appendix A, 'Tensor Convolution'):
for a convolved label held by a feature operand (size I) and a filter operand
(size K),   out[p] = sum_k feat[p + k - c] * filt[k],   c = floor((K-1)/2),
with feat zero outside [0, I) and p in [0, I): cross-correlation, stride 1,
same padding (the output keeps the feature size).
"""
from __future__ import annotations

import itertools

import numpy as np

from .cost import kept_labels, label_size, stride_of, is_circular
from .notation import Expr


def _letters(expr: Expr):
    pool = "abcdefghijklmnopqrstuvwxyzABCDEFGHIJKLMNOPQRSTUVWXYZ"
    labs = expr.all_labels()
    if len(labs) > len(pool):
        raise ValueError("too many labels for numpy.einsum")
    return {l: pool[i] for i, l in enumerate(labs)}


def _einsum(letters, a, la, b, lb, lc):
    sub = "".join(letters[l] for l in la) + "," + "".join(letters[l] for l in lb) + \
        "->" + "".join(letters[l] for l in lc)
    return np.einsum(sub, a, b, optimize=True)


def shift(a, axis, tap, K, stride=1):
    """out[p] = a[stride*p + tap - floor((K-1)/2)] for p in [0, ceil(n/stride))
    (zero where that index leaves the array): the feature operand as seen by
    filter tap `tap`."""
    n = a.shape[axis]
    m = -(-n // stride)
    p = np.arange(m)
    q = stride * p + tap - (K - 1) // 2
    ok = (q >= 0) & (q < n)
    shape = list(a.shape)
    shape[axis] = m
    out = np.zeros(shape, dtype=np.float64)
    dst = [slice(None)] * a.ndim
    dst[axis] = p[ok]
    out[tuple(dst)] = np.take(a, q[ok], axis=axis)
    return out


def shift_adjoint(g, axis, tap, K, n=None, stride=1):
    """Adjoint of shift() for a feature of length n (default: g's length):
    out[stride*p + tap - floor((K-1)/2)] = g[p] where that index lies in
    [0, n), zero elsewhere (distinct p give distinct positions)."""
    m = g.shape[axis]
    n = m if n is None else n
    p = np.arange(m)
    q = stride * p + tap - (K - 1) // 2
    ok = (q >= 0) & (q < n)
    shape = list(g.shape)
    shape[axis] = n
    out = np.zeros(shape, dtype=np.float64)
    dst = [slice(None)] * g.ndim
    dst[axis] = q[ok]
    out[tuple(dst)] = np.take(g, p[ok], axis=axis)
    return out


def circ_shift(a, axis, tap, N):
    """out[p] = a[(p - tap) mod N] for p in [0, N), a zero-padded to length N:
    the side of a circular convolution as seen by position `tap` of the other
    side."""
    n = a.shape[axis]
    q = (np.arange(N) - tap) % N
    ok = q < n
    shape = list(a.shape)
    shape[axis] = N
    out = np.zeros(shape, dtype=np.float64)
    dst = [slice(None)] * a.ndim
    dst[axis] = np.arange(N)[ok]
    out[tuple(dst)] = np.take(a, q[ok], axis=axis)
    return out


def circ_shift_adjoint(g, axis, tap, N, n):
    """Adjoint of circ_shift() for a side of length n: out[i] = g[(i + tap)
    mod N], i in [0, n)."""
    return np.take(g, (np.arange(n) + tap) % N, axis=axis)


def step_convs(expr: Expr, A, B):
    """Convolved labels performed by the step merging operand sets A and B:
    [(label, feature on A?)] for linear labels, [(label, None)] for circular
    ones (taps over side B)."""
    la, lb = kept_labels(expr, A), kept_labels(expr, B)
    res = []
    for l in la:
        if l in lb and l in expr.conv:
            if is_circular(expr, l):
                res.append((l, None))
            else:
                res.append((l, expr.feature[l] in set(A)))
    return res


def pair_step(expr, letters, a, A, b, B):
    """One pairwise step: tensors a (operand set A) and b (operand set B),
    each in kept-label order, to the merged tensor in kept-label order."""
    la, lb = kept_labels(expr, A), kept_labels(expr, B)
    lc = kept_labels(expr, tuple(A) + tuple(B))
    convs = step_convs(expr, A, B)
    taps = []
    for l, fa in convs:
        K = label_size(expr, B, l) if fa or fa is None else label_size(expr, A, l)
        taps.append(range(K))
    acc = None
    for combo in itertools.product(*taps):
        xa, xb, ca, cb = a, b, list(la), list(lb)
        for (l, fa), k in zip(convs, combo):
            if fa is None:
                # circular: side A at (p - k) mod N against position k of side B
                N = label_size(expr, tuple(A) + tuple(B), l)
                xa = circ_shift(xa, ca.index(l), k, N)
                xb = np.take(xb, k, axis=cb.index(l))
                cb.remove(l)
            elif fa:
                K = label_size(expr, B, l)
                xa = shift(xa, ca.index(l), k, K, stride_of(expr, l))
                xb = np.take(xb, k, axis=cb.index(l))
                cb.remove(l)
            else:
                K = label_size(expr, A, l)
                xb = shift(xb, cb.index(l), k, K, stride_of(expr, l))
                xa = np.take(xa, k, axis=ca.index(l))
                ca.remove(l)
        term = _einsum(letters, xa, ca, xb, cb, lc)
        acc = term if acc is None else acc + term
    return acc, lc


def leaf_tensor(expr, arrays, i):
    """Operand i with its self-contracted labels summed away (Section 3.1,
    case (5)): labels held by operand i only and absent from the output."""
    li = list(expr.inputs[i])
    keep = kept_labels(expr, (i,))
    a = np.asarray(arrays[i], dtype=np.float64)
    drop = tuple(k for k, l in enumerate(li) if l not in keep)
    if drop:
        a = a.sum(axis=drop)
    rest = [l for l in li if l in keep]
    return np.transpose(a, [rest.index(l) for l in keep]), keep


def eval_pairwise(expr: Expr, arrays, tree, keep_intermediates: bool = False):
    """Evaluate along `tree` (nested pairs of operand indices)."""
    letters = _letters(expr)
    inter = {}

    def rec(t):
        if isinstance(t, int):
            a, _ = leaf_tensor(expr, arrays, t)
            return a, (t,)
        a, A = rec(t[0])
        b, B = rec(t[1])
        c, _ = pair_step(expr, letters, a, A, b, B)
        if keep_intermediates:
            inter[tuple(sorted(A + B))] = c
        return c, A + B

    if isinstance(tree, int):
        a, _ = leaf_tensor(expr, arrays, tree)
        res, lres = a, kept_labels(expr, (tree,))
    else:
        res, S = rec(tree)
        lres = kept_labels(expr, S)
    perm = [lres.index(l) for l in expr.output]
    y = np.transpose(res, perm).copy()
    return (y, inter) if keep_intermediates else y


def eval_definition(expr: Expr, arrays):
    """Y[o] = sum over every label not in the output and over the taps of
    each convolved label of the product of all operands' entries; the feature
    operand of a convolved label is read at s*p + k - c (zero outside; s the
    label's stride, 1 unless given), its filter operand at tap k, the output
    at p; a circular label's holders are read at positions summing to p
    modulo N (zero past a holder's size)."""
    conv2 = {l: expr.feature[l] for l in expr.conv if l in expr.feature}
    # circular labels: the first holder is read at (p - sum of the other
    # holders' positions) mod N, the others at every position
    circ = [l for l in expr.conv if is_circular(expr, l)]
    first = {l: expr.holders(l)[0] for l in circ}
    N = {l: expr.out_sizes[l] for l in circ}
    ctaps = [(l, i) for l in circ for i in expr.holders(l)[1:]]
    K = {}
    for l, f in conv2.items():
        other = [i for i in expr.holders(l) if i != f][0]
        K[l] = expr.sizes[other][l]
    out_shape = tuple(expr.out_sizes[l] for l in expr.output)
    red = [l for l in expr.all_labels() if l not in expr.output]
    red_size = {}
    for l in red:
        red_size[l] = expr.sizes[expr.holders(l)[0]][l]
    y = np.zeros(out_shape)
    arrs = [np.asarray(a, dtype=np.float64) for a in arrays]
    for o in itertools.product(*[range(d) for d in out_shape]):
        ov = dict(zip(expr.output, o))
        s = 0.0
        for r in itertools.product(*[range(red_size[l]) for l in red]):
            rv = dict(zip(red, r))
            for kk in itertools.product(*[range(K[l]) for l in conv2],
                                        *[range(expr.sizes[i][l]) for l, i in ctaps]):
                kv = dict(zip(conv2, kk))
                cv = dict(zip(ctaps, kk[len(conv2):]))
                prod = 1.0
                for i, labs in enumerate(expr.inputs):
                    idx = []
                    for l in labs:
                        if l in first:
                            if i == first[l]:
                                pos = (ov[l] - sum(cv[(l, j)] for j in expr.holders(l)[1:])) % N[l]
                                if pos >= expr.sizes[i][l]:
                                    prod = 0.0
                                    break
                                idx.append(pos)
                            else:
                                idx.append(cv[(l, i)])
                        elif l in conv2:
                            if i == conv2[l]:
                                pos = stride_of(expr, l) * ov[l] + kv[l] - (K[l] - 1) // 2
                                if pos < 0 or pos >= expr.sizes[i][l]:
                                    prod = 0.0
                                    break
                                idx.append(pos)
                            else:
                                idx.append(kv[l])
                        elif l in ov:
                            idx.append(ov[l])
                        else:
                            idx.append(rv[l])
                    if prod == 0.0:
                        break
                    prod *= arrs[i][tuple(idx)]
                s += prod
        y[o] = s
    return y


def dense_kernel(expr: Expr, arrays, feature_operand: int = 0):
    """Merge every operand except the feature operand into one dense kernel
    (a plain einsum: no label of the factors is convolved against another
    factor).  Returns (W, labels of W)."""
    others = [i for i in range(expr.n) if i != feature_operand]
    for l in expr.conv:
        if len(expr.holders(l)) != 2 or expr.feature.get(l) != feature_operand:
            raise NotImplementedError(
                "dense evaluation needs every convolved label on the feature operand "
                "and exactly one factor")
    lw = kept_labels(expr, others)
    letters = _letters(expr)
    sub = ",".join("".join(letters[l] for l in expr.inputs[i]) for i in others) + \
        "->" + "".join(letters[l] for l in lw)
    W = np.einsum(sub, *[np.asarray(arrays[i], np.float64) for i in others], optimize=True)
    return W, lw


def eval_dense(expr: Expr, arrays, feature_operand: int = 0):
    """Y = X (*) W_dense: zero-pad X along each convolved label, then add one
    einsum per filter tap over the shifted window (every s-th position for a
    label of stride s)."""
    W, lw = dense_kernel(expr, arrays, feature_operand)
    X = np.asarray(arrays[feature_operand], np.float64)
    lx = list(expr.inputs[feature_operand])
    keep_x = kept_labels(expr, (feature_operand,))
    drop = tuple(k for k, l in enumerate(lx) if l not in keep_x)
    if drop:
        X = X.sum(axis=drop)
        lx = keep_x
    convs = [l for l in expr.conv]
    Ks = [W.shape[lw.index(l)] for l in convs]
    pads = [(0, 0)] * X.ndim
    for l, K in zip(convs, Ks):
        c = (K - 1) // 2
        pads[lx.index(l)] = (c, K - 1 - c)
    Xp = np.pad(X, pads)
    letters = _letters(expr)
    Y = None
    lw_red = [l for l in lw if l not in convs]
    for combo in itertools.product(*[range(K) for K in Ks]):
        win = [slice(None)] * X.ndim
        widx = [slice(None)] * W.ndim
        for l, k in zip(convs, combo):
            # padded position s*p + k for the output positions p
            s = stride_of(expr, l)
            m = expr.out_sizes[l]
            win[lx.index(l)] = slice(k, k + s * (m - 1) + 1, s)
            widx[lw.index(l)] = k
        term = _einsum(letters, Xp[tuple(win)], lx, W[tuple(widx)], lw_red, expr.output)
        Y = term if Y is None else Y + term
    return Y
