"""conv_einsum strings and size binding (test infrastructure; see package doc).

Grammar, from Section 2.2 ('From einsum to conv_einsum') and the layer
strings of Appendix A.3:

    spec   := terms '->' term [ '|' convs ]
    terms  := term ( ',' term )*
    term   := label*
    label  := a single letter  |  '(' name ')'        e.g. (s1), (r0)
    convs  := label ( [','] label )*                  e.g. |hw  or  |h,w

Blanks are ignored.  A label may occur at most once per operand and once in
the output.  A label that is not convolved must have one size everywhere
(Appendix A, contraction: the method fails when sizes of the same letter
differ); a convolved label may carry a different size in each operand
(Section 2.2 lets one letter name convolved modes of unequal sizes, such as
an image axis and the filter axis it is convolved with).
"""
from __future__ import annotations

from dataclasses import dataclass


def _labels(term: str, where: str):
    out, i = [], 0
    while i < len(term):
        c = term[i]
        if c == "(":
            j = term.find(")", i)
            if j < 0:
                raise ValueError(f"unclosed '(' in {where}")
            name = term[i + 1:j]
            if not name or not all(ch.isalnum() or ch == "_" for ch in name):
                raise ValueError(f"bad label '({name})' in {where}")
            out.append(name)
            i = j + 1
        elif c.isalpha():
            out.append(c)
            i += 1
        else:
            raise ValueError(f"unexpected character {c!r} in {where}")
    return out


@dataclass
class Expr:
    inputs: list            # list of label lists, one per operand
    output: list            # output label list
    conv: list              # convolved labels, in the order written after '|'
    sizes: list = None      # per operand: {label: size}; set by bind()
    feature: dict = None    # conv label -> operand index of its feature side
    out_sizes: dict = None  # output label -> size
    stride: dict = None     # conv label -> stride (absent: 1)
    circular: set = None    # conv labels convolved circularly (commutative)

    @property
    def n(self):
        return len(self.inputs)

    def all_labels(self):
        seen = []
        for t in self.inputs:
            for l in t:
                if l not in seen:
                    seen.append(l)
        return seen

    def holders(self, label):
        return [i for i, t in enumerate(self.inputs) if label in t]


def parse(spec: str) -> Expr:
    s = "".join(spec.split())
    if s.count("->") != 1:
        raise ValueError("a conv_einsum string needs exactly one '->'")
    lhs, rhs = s.split("->")
    if "|" in rhs:
        if rhs.count("|") != 1:
            raise ValueError("at most one '|'")
        out_s, conv_s = rhs.split("|")
    else:
        out_s, conv_s = rhs, ""
    if "|" in lhs:
        raise ValueError("'|' must follow the output term")
    terms = lhs.split(",")
    inputs = [_labels(t, f"operand {i}") for i, t in enumerate(terms)]
    for i, t in enumerate(inputs):
        if len(set(t)) != len(t):
            raise ValueError(f"operand {i} repeats a label")
    output = _labels(out_s, "output")
    if len(set(output)) != len(output):
        raise ValueError("output repeats a label")
    conv = []
    for piece in conv_s.split(","):
        for l in _labels(piece, "convolution list"):
            if l in conv:
                raise ValueError(f"convolved label {l} listed twice")
            conv.append(l)
    present = {l for t in inputs for l in t}
    for l in output:
        if l not in present:
            raise ValueError(f"output label {l} is in no operand")
    for l in conv:
        if l not in present:
            raise ValueError(f"convolved label {l} is in no operand")
        if l not in output:
            raise ValueError(f"convolved label {l} must be kept in the output")
    return Expr(inputs=inputs, output=output, conv=conv)


def bind(expr: Expr, shapes, feature_operand: int = 0, strides=None, circular=()) -> Expr:
    """Attach operand sizes and resolve the feature side of each convolved label.

    Feature side (Appendix B, 'Convolution Varieties'): of the two operands
    holding a convolved label, the one with the larger size holds features and
    the other holds filters.  On equal sizes the designated feature operand
    wins if it is one of the two, otherwise the operand with the lower index.
    A convolved label held by more than two operands is multi-way; it is kept
    (its cost is defined) but has no feature side.

    `strides` maps a convolved label held by two operands to its stride s >= 1
    (a strided convolution is one of the non-commutative varieties of
    Appendix B): output position p reads the feature at s*p + k - c, and the
    output keeps ceil(I / s) positions (I = feature size).

    Circular convolution (Appendix B: the only kind supported for a label held
    by more than two operands, and commutative): every holder is zero-padded
    to N, the largest of its sizes, and indices add modulo N,
        out[p] = sum over i_1 + ... + i_m = p (mod N) of prod_k T_k[i_k],
    p in [0, N).  Labels held by three or more operands are circular; a
    two-way label is circular when listed in `circular` (then it has no
    feature side).
    """
    if len(shapes) != expr.n:
        raise ValueError("one shape per operand is required")
    sizes = []
    for i, (t, shp) in enumerate(zip(expr.inputs, shapes)):
        shp = tuple(int(d) for d in shp)
        if len(shp) != len(t):
            raise ValueError(f"operand {i}: rank {len(shp)} != {len(t)} labels")
        if any(d < 1 for d in shp):
            raise ValueError(f"operand {i}: sizes must be >= 1")
        sizes.append(dict(zip(t, shp)))
    common = {}
    for i, sz in enumerate(sizes):
        for l, d in sz.items():
            if l in expr.conv:
                continue
            if l in common and common[l] != d:
                raise ValueError(f"label {l}: size {d} in operand {i} != {common[l]}")
            common[l] = d
    circ = set()
    for l in expr.conv:
        if len(expr.holders(l)) > 2:
            circ.add(l)
    for l in circular or ():
        if l not in expr.conv or len(expr.holders(l)) < 2:
            raise ValueError(f"circular {l}: a convolved label held by two or more operands")
        circ.add(l)
    feature = {}
    for l in expr.conv:
        hold = expr.holders(l)
        if len(hold) == 2 and l not in circ:
            a, b = hold
            da, db = sizes[a][l], sizes[b][l]
            if da != db:
                feature[l] = a if da > db else b
            elif feature_operand in (a, b):
                feature[l] = feature_operand
            else:
                feature[l] = min(a, b)
    stride = {}
    for l, st in (strides or {}).items():
        if l not in feature:
            raise ValueError(f"stride of {l}: only a convolved label held by two operands is strided")
        if int(st) < 1:
            raise ValueError(f"stride of {l} must be >= 1")
        if int(st) > 1:
            stride[l] = int(st)
    out_sizes = {}
    for l in expr.output:
        if l in feature:            # same padding keeps the feature size (ceil(I / s) when strided)
            s_ = stride.get(l, 1)
            out_sizes[l] = -(-sizes[feature[l]][l] // s_)
        elif l in expr.conv:        # one holder, or circular: the largest size N
            out_sizes[l] = max(sizes[i][l] for i in expr.holders(l))
        else:
            out_sizes[l] = common[l]
    expr.sizes = sizes
    expr.feature = feature
    expr.out_sizes = out_sizes
    expr.stride = stride
    expr.circular = circ
    return expr
