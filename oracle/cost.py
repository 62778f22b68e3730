"""tnn-cost: multiplications of a pairwise step (test infrastructure).

Appendix B lists the cost of each primitive between T0 (sizes I_p) and T1
(sizes J_q): a contraction or batch product costs prod(I) * prod(J without
the shared mode), an outer product prod(I) * prod(J), and a convolution
(no FFT) prod(I) * prod(J).  A pairwise step of conv_einsum mixes these
primitives; counting each multiplication once gives the reading used here:

    cost = prod over the union of the two operands' labels of the label size,
           where a label shared by both operands counts once, except a
           convolved label held by both, which counts I * J (feature size
           times filter size).

The worked costs of Appendix B (2-D convolution: BHWXYTS) and of the proof of
Theorem 1 (BRTHWH'W', BSTHWH'W') are instances of this rule.

Operands of a step are intermediate tensors.  The labels an intermediate keeps
are the labels of its operands that are in the output or still held by an
operand outside it.  A label held by a single operand and absent from the
output (self-contraction, Section 3.1 case (5)) is summed away before any
pairwise step, so it never enters a step cost.  A convolved label's size in an
intermediate is the largest size among the operands it merges (the feature
size once the convolution has been done).

Training mode (Appendix B, 'Modification of the cost model for training'):
cost(f) + cost(g1) + cost(g2), with g1, g2 the gradients with respect to the
two operands, costed by the same equations.  For the gradient of the feature
side a convolved label counts (output size) * (filter size); for the
gradient of the filter side it counts (feature size) * (output size), as in
the Appendix B example cost(g1) = BHWX'Y'TS, cost(g2) = BXYX'Y'TS.  With
same padding the output size equals the feature size.

A circular label (Appendix B: multi-way labels are convolved circularly)
counts a * b in a step merging sides of sizes a and b (every pair of
positions meets once, in the forward and in each gradient), and a tensor
that merges two or more of its holders holds its N positions.

A strided convolved label (stride s) has ceil(I / s) output positions; a step
that convolves it counts (output size) * (filter size), the multiplications
it does (I * J for s = 1), and the merged tensor holds the output size.
"""
from __future__ import annotations

from .notation import Expr


def kept_labels(expr: Expr, subset):
    """Labels of the intermediate tensor that merges the operands in `subset`,
    in order of first appearance in the string."""
    sub = set(subset)
    res = []
    for l in expr.all_labels():
        held_in = [i for i in expr.holders(l) if i in sub]
        if not held_in:
            continue
        outside = [i for i in expr.holders(l) if i not in sub]
        if l in expr.output or outside:
            res.append(l)
    return res


def stride_of(expr: Expr, label) -> int:
    return (expr.stride or {}).get(label, 1)


def is_circular(expr: Expr, label) -> bool:
    return label in (expr.circular or ())


def label_size(expr: Expr, subset, label):
    """Size of `label` in the tensor merging the operands in `subset`: the
    largest size among them, except a strided convolved label once both of
    its holders are merged, which has ceil(I / s) output positions, and a
    circular label once two or more of its holders are merged, which has the
    N positions of the circular convolution (its largest size overall)."""
    if is_circular(expr, label):
        hold = expr.holders(label)
        if sum(1 for i in hold if i in subset) >= 2:
            return max(expr.sizes[i][label] for i in hold)
    s = stride_of(expr, label)
    if s > 1 and all(i in subset for i in expr.holders(label)):
        return -(-expr.sizes[expr.feature[label]][label] // s)
    return max(expr.sizes[i][label] for i in subset if label in expr.inputs[i])


def _feature_side_is_a(expr: Expr, A, B, l):
    if l in expr.feature:
        return expr.feature[l] in A
    # multi-way label: the larger size is treated as the feature side
    return label_size(expr, A, l) >= label_size(expr, B, l)


def step_cost(expr: Expr, A, B, mode: str = "fwd") -> int:
    """Multiplications of the pairwise step merging operand sets A and B."""
    A, B = set(A), set(B)
    la, lb = kept_labels(expr, A), kept_labels(expr, B)
    plain = 1
    both = []          # (feature size, filter size, feature on A?, output size)
    circ = 1           # circular labels: every pair of positions once
    for l in la + [x for x in lb if x not in la]:
        if l in la and l in lb and is_circular(expr, l):
            circ *= label_size(expr, A, l) * label_size(expr, B, l)
        elif l in la and l in lb and l in expr.conv:
            ia, ib = label_size(expr, A, l), label_size(expr, B, l)
            if _feature_side_is_a(expr, A, B, l):
                both.append((ia, ib, True, -(-ia // stride_of(expr, l))))
            else:
                both.append((ib, ia, False, -(-ib // stride_of(expr, l))))
        elif l in la:
            plain *= label_size(expr, A, l)
        else:
            plain *= label_size(expr, B, l)
    plain *= circ
    f = plain
    for feat, filt, _, out in both:
        f *= out * filt
    if mode == "fwd":
        return f
    if mode != "train_paper":
        raise ValueError(mode)
    ga = plain   # gradient w.r.t. the operand on side A
    gb = plain
    for feat, filt, fa, out in both:
        if fa:
            ga *= out * filt
            gb *= feat * out
        else:
            ga *= feat * out
            gb *= out * filt
    return f + ga + gb


def _leaves(t):
    return (t,) if isinstance(t, int) else _leaves(t[0]) + _leaves(t[1])


def step_costs(expr: Expr, tree, mode: str = "fwd"):
    """Per-step costs of a tree, in post order (left child first)."""
    out = []

    def rec(t):
        if isinstance(t, int):
            return
        rec(t[0])
        rec(t[1])
        out.append(step_cost(expr, _leaves(t[0]), _leaves(t[1]), mode))

    rec(tree)
    return out


def tree_cost(expr: Expr, tree, mode: str = "fwd") -> int:
    return sum(step_costs(expr, tree, mode))
