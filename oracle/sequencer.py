"""Brute-force optimal sequencer (test infrastructure).

Section 3.2 evaluates an N-operand conv_einsum as a sequence of pairwise
steps and picks the sequence with the fewest multiplications under tnn-cost.
The oracle enumerates every full binary tree over the operands (outer products
included) and keeps the cheapest.

Trees are nested pairs of operand indices; in each pair the first child is
the one holding the lowest operand index.  When several trees share the
minimum cost the paper does not say which one is returned; the reading used
here is the lexicographically smallest key

    key(leaf) = ()
    key((L, R)) = (bitmask of L's operands, key(L), key(R))

which a subset dynamic programme reproduces by always taking, among the
cheapest splits of a set, the split whose first part has the smallest
bitmask.  Steps execute in post order, first child first.
"""
from __future__ import annotations

import itertools

from .cost import kept_labels, label_size, step_cost


def leaves(t):
    return (t,) if isinstance(t, int) else leaves(t[0]) + leaves(t[1])


def _mask(t):
    m = 0
    for i in leaves(t):
        m |= 1 << i
    return m


def key(t):
    if isinstance(t, int):
        return ()
    return (_mask(t[0]), key(t[0]), key(t[1]))


def all_trees(ops):
    """Every full binary tree over the operand indices in `ops`."""
    ops = tuple(sorted(ops))
    if len(ops) == 1:
        yield ops[0]
        return
    first, rest = ops[0], ops[1:]
    for r in range(len(rest)):
        for comb in itertools.combinations(rest, r):
            a = (first,) + comb
            b = tuple(o for o in rest if o not in comb)
            for ta in all_trees(a):
                for tb in all_trees(b):
                    yield (ta, tb)


def count_trees(n):
    """(2n-3)!! full binary trees over n labelled leaves."""
    c = 1
    for k in range(1, 2 * n - 2, 2):
        c *= k
    return c


def intermediate_size(expr, subset) -> int:
    """Elements of the tensor that merges the operands in `subset`: the
    product of the sizes of its kept labels (a convolved label at its largest
    size among the merged operands)."""
    n = 1
    for l in kept_labels(expr, subset):
        n *= label_size(expr, subset, l)
    return n


def max_intermediate(expr, t) -> int:
    """Largest intermediate of tree t (its internal nodes except the root,
    which is the output); 0 for a single step or a leaf."""
    sizes = []

    def rec(x, root):
        if isinstance(x, int):
            return
        if not root:
            sizes.append(intermediate_size(expr, leaves(x)))
        rec(x[0], False)
        rec(x[1], False)

    rec(t, True)
    return max(sizes, default=0)


def optimal_tree(expr, mode: str = "fwd", return_all: bool = False, max_elements=None,
                 max_step_cost=None):
    """Cheapest tree by exhaustive search, ties broken by the smallest key.

    With `max_step_cost`, only trees in which every pairwise step (every
    internal node) costs at most that much under `mode` compete: the path
    that meets a user-given cost cap at each node (Section 3.2, Figure 2,
    the orange path).  With `max_elements`, only trees whose every
    intermediate holds at most that many elements compete (a memory limit on
    the intermediates, the other reading of the same trade-off).
    (None, None) when no tree qualifies."""
    memo = {}

    def sc(a, b):
        k = (a, b)
        if k not in memo:
            memo[k] = step_cost(expr, leaves_of_mask(a), leaves_of_mask(b), mode)
        return memo[k]

    def cost(t):
        if isinstance(t, int):
            return 0
        return cost(t[0]) + cost(t[1]) + sc(_mask(t[0]), _mask(t[1]))

    def steps_within(t):
        if isinstance(t, int):
            return True
        return (sc(_mask(t[0]), _mask(t[1])) <= max_step_cost and steps_within(t[0])
                and steps_within(t[1]))

    best, best_cost, ties = None, None, []
    for t in all_trees(range(expr.n)):
        if max_elements is not None and max_intermediate(expr, t) > max_elements:
            continue
        if max_step_cost is not None and not steps_within(t):
            continue
        c = cost(t)
        if best_cost is None or c < best_cost:
            best, best_cost, ties = t, c, [t]
        elif c == best_cost:
            ties.append(t)
            if key(t) < key(best):
                best = t
    if return_all:
        return best, best_cost, ties
    return best, best_cost


def leaves_of_mask(m):
    out, i = [], 0
    while m:
        if m & 1:
            out.append(i)
        m >>= 1
        i += 1
    return tuple(out)


def left_to_right_tree(n):
    """((((0,1),2),3),...): operands paired in string order (Section 3.2,
    'Better than left-to-right evaluation'; the naive baseline of Section 5)."""
    t = 0
    for i in range(1, n):
        t = (t, i)
    return t


def tree_from_pairs(n, pairs):
    """Tree from a list of (i, j) positions in the current operand list; the
    merged tensor is appended to the end of the list (opt_einsum's path
    format)."""
    cur = list(range(n))
    for i, j in pairs:
        if i == j or not (0 <= i < len(cur)) or not (0 <= j < len(cur)):
            raise ValueError("bad pair")
        a, b = cur[i], cur[j]
        for k in sorted((i, j), reverse=True):
            del cur[k]
        node = (a, b) if min(leaves(a)) < min(leaves(b)) else (b, a)
        cur.append(node)
    if len(cur) != 1:
        raise ValueError("pairs do not merge every operand")
    return cur[0]


def post_order_steps(t):
    """[(left, right), ...] in execution order."""
    out = []

    def rec(x):
        if isinstance(x, int):
            return
        rec(x[0])
        rec(x[1])
        out.append((x[0], x[1]))

    rec(t)
    return out


def checkpoint_choice(expr, tree, budget_bytes: int, elem_bytes: int, mode: str = "fwd"):
    """Which intermediates to keep from the forward for the backward
    (Section 3.3: keeping intermediates costs memory, recomputing them costs
    multiplications).  Every intermediate (every step result but the last) is
    a candidate; keeping the result of step s spares its recompute, step_cost
    of that step.  Returns (set of kept step indices in post order, kept
    bytes, multiplications still recomputed): the subset with the largest
    spared cost whose bytes (elements x elem_bytes) fit the budget; ties go
    to fewer bytes, then to the smaller bitmask of step indices."""
    steps = post_order_steps(tree)
    costs = []
    sizes = []
    for a, b in steps[:-1]:
        la, lb = leaves(a), leaves(b)
        costs.append(step_cost(expr, la, lb, mode))
        sizes.append(intermediate_size(expr, tuple(la) + tuple(lb)) * elem_bytes)
    best = None
    for mask in range(1 << len(costs)):
        kept = [s for s in range(len(costs)) if (mask >> s) & 1]
        w = sum(sizes[s] for s in kept)
        if w > budget_bytes:
            continue
        v = sum(costs[s] for s in kept)
        key_ = (-v, w, mask)
        if best is None or key_ < best[0]:
            best = (key_, set(kept), w, sum(costs) - v)
    return best[1], best[2], best[3]
