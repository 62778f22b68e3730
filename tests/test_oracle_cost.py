"""Pins for tnn-cost and the optimal sequencer (CPU).

Closed forms come from the paper (Appendix B primitive costs and the 2-D
convolution training example; the proof of Theorem 1), the tree count and the
matrix-chain optimum from textbooks."""
import itertools
import random

import pytest

import oracle as O


def _e(spec, shapes, **kw):
    return O.bind(O.parse(spec), shapes, **kw)


def test_primitive_costs_appendix_b():
    # contraction over a: prod(I) * prod(J without the shared mode)
    A, B, C, D, E = 3, 4, 5, 6, 7
    e = _e("abc,ade->bcde", [(A, B, C), (A, D, E)])
    assert O.step_cost(e, (0,), (1,)) == (A * B * C) * (D * E)
    # outer product: prod(I) * prod(J)
    e = _e("abc,def->abcdef", [(A, B, C), (D, E, 2)])
    assert O.step_cost(e, (0,), (1,)) == (A * B * C) * (D * E * 2)
    # batch product over c: prod(I) * prod(J without the shared mode)
    e = _e("abc,cde->abcde", [(A, B, C), (C, D, E)])
    assert O.step_cost(e, (0,), (1,)) == (A * B * C) * (D * E)
    # convolution (no FFT): prod(I) * prod(J)
    X, L = 11, 3
    e = _e("xbc,xde->xbcde|x", [(X, B, C), (L, D, E)])
    assert O.step_cost(e, (0,), (1,)) == (X * B * C) * (L * D * E)


@pytest.mark.parametrize("Bn,S,T,X,Y,H,W", [(2, 3, 4, 9, 7, 3, 3), (5, 2, 3, 16, 11, 5, 2)])
def test_2d_conv_forward_and_training_cost(Bn, S, T, X, Y, H, W):
    """Appendix B: cost(f) = BHWXYTS, cost(g1) = BHWX'Y'TS, cost(g2) =
    BXYX'Y'TS, with X' = X, Y' = Y under same padding."""
    e = _e("bsxy,tsxy->btxy|xy", [(Bn, S, X, Y), (T, S, H, W)])
    f = Bn * H * W * X * Y * T * S
    g1 = Bn * H * W * X * Y * T * S
    g2 = Bn * X * Y * X * Y * T * S
    assert O.step_cost(e, (0,), (1,)) == f
    assert O.step_cost(e, (0,), (1,), "train_paper") == f + g1 + g2
    # the filter may be written first: the costs do not depend on the order
    e2 = _e("tsxy,bsxy->btxy|xy", [(T, S, H, W), (Bn, S, X, Y)])
    assert O.step_cost(e2, (0,), (1,), "train_paper") == f + g1 + g2


def _rcp(M, Bn, R, Ss, Ts, Hp, Wp, H, W):
    ops = ["b" + "".join(f"(s{i+1})" for i in range(M)) + "hw"]
    shapes = [(Bn,) + tuple(Ss) + (Hp, Wp)]
    for i in range(M):
        ops.append(f"r(t{i+1})(s{i+1})")
        shapes.append((R, Ts[i], Ss[i]))
    ops.append("rhw")
    shapes.append((R, H, W))
    out = "b" + "".join(f"(t{i+1})" for i in range(M)) + "hw"
    return _e(",".join(ops) + "->" + out + "|hw", shapes)


def _prod(xs):
    p = 1
    for x in xs:
        p *= x
    return p


def _theorem1_cases(n=30, seed=0):
    rnd = random.Random(seed)
    for _ in range(n):
        M = rnd.choice([2, 3, 4])
        Ss = [rnd.randint(1, 4) for _ in range(M)]
        Ts = [rnd.randint(1, 4) for _ in range(M)]
        yield M, rnd.randint(1, 6), rnd.randint(1, 9), Ss, Ts, rnd.randint(5, 30), \
            rnd.randint(5, 30), rnd.choice([1, 3, 5]), rnd.choice([1, 3, 5])


@pytest.mark.parametrize("case", list(_theorem1_cases()))
def test_theorem1_left_to_right_cost(case):
    """Proof of Theorem 1: M_naive = B R H'W' sum_i U_i + B R T H W H'W' with
    U_k = prod_{i>=k} S_i prod_{i<=k} T_i.  The printed U_M = T drops S_M,
    which the last mode product still contracts; S_M T is used."""
    M, Bn, R, Ss, Ts, Hp, Wp, H, W = case
    e = _rcp(M, Bn, R, Ss, Ts, Hp, Wp, H, W)
    T = _prod(Ts)
    U = [_prod(Ss[k:]) * _prod(Ts[:k + 1]) for k in range(M)]
    naive = Bn * R * Hp * Wp * sum(U) + Bn * R * T * H * W * Hp * Wp
    assert O.tree_cost(e, O.left_to_right_tree(M + 2)) == naive


@pytest.mark.parametrize("case", list(_theorem1_cases()))
def test_theorem1_reduced_path_cost(case):
    """Proof of Theorem 1: merging W1..WM, then W0, then convolving with X
    costs R sum_{i>=2} V_i + R S T H W + B S T H W H'W', V_k = prod_{i<=k} S_i T_i
    (the printed sum from i = 1 counts R S1 T1 for W1 alone, which is no
    operation)."""
    M, Bn, R, Ss, Ts, Hp, Wp, H, W = case
    e = _rcp(M, Bn, R, Ss, Ts, Hp, Wp, H, W)
    S, T = _prod(Ss), _prod(Ts)
    V = [_prod(Ss[:k + 1]) * _prod(Ts[:k + 1]) for k in range(M)]
    reduced = R * sum(V[1:]) + R * S * T * H * W + Bn * S * T * H * W * Hp * Wp
    merged = 1
    for i in range(2, M + 1):
        merged = (merged, i)
    tree = (0, (merged, M + 1))
    assert O.tree_cost(e, tree) == reduced


def test_theorem1_claim_optimal_beats_left_to_right():
    """Theorem 1: with H'W' >> HW (S H'W' > aHW, B H'W' > aS) and R >= S a
    path cheaper than left-to-right exists, so the optimum is cheaper."""
    rnd = random.Random(1)
    checked = 0
    while checked < 15:
        M = 3
        Ss = [rnd.randint(1, 3) for _ in range(M)]
        Ts = [rnd.randint(1, 3) for _ in range(M)]
        S = _prod(Ss)
        R = rnd.randint(S, S + 6)
        Bn, Hp, Wp, H, W = rnd.randint(1, 4), rnd.randint(8, 20), rnd.randint(8, 20), 3, 3
        if not (S * Hp * Wp > H * W and Bn * Hp * Wp > S):
            continue
        e = _rcp(M, Bn, R, Ss, Ts, Hp, Wp, H, W)
        _, best = O.optimal_tree(e)
        assert best < O.tree_cost(e, O.left_to_right_tree(M + 2))
        checked += 1


def test_theorem2_claim_tucker():
    """Theorem 2 (reshaped Tucker): with prod R_m >= S the optimum is cheaper
    than left-to-right."""
    rnd = random.Random(2)
    for _ in range(6):
        Ss = [rnd.randint(1, 3) for _ in range(3)]
        Ts = [rnd.randint(1, 3) for _ in range(3)]
        Rs = [rnd.randint(1, 3) for _ in range(4)]
        while Rs[1] * Rs[2] * Rs[3] < _prod(Ss):
            Rs[rnd.randint(1, 3)] += 1
        Bn, Hp, Wp = 2, rnd.randint(8, 14), rnd.randint(8, 14)
        spec = ("b(s1)(s2)(s3)hw,(r1)(t1)(s1),(r2)(t2)(s2),(r3)(t3)(s3),(r0)hw,"
                "(r0)(r1)(r2)(r3)->b(t1)(t2)(t3)hw|hw")
        shapes = [(Bn, *Ss, Hp, Wp), (Rs[1], Ts[0], Ss[0]), (Rs[2], Ts[1], Ss[1]),
                  (Rs[3], Ts[2], Ss[2]), (Rs[0], 3, 3), tuple(Rs)]
        e = _e(spec, shapes)
        _, best = O.optimal_tree(e)
        assert best < O.tree_cost(e, O.left_to_right_tree(6))


@pytest.mark.parametrize("n", range(1, 8))
def test_tree_count_is_double_factorial(n):
    assert sum(1 for _ in O.all_trees(range(n))) == O.count_trees(n)
    if n >= 2:
        assert O.count_trees(n) == _prod(range(1, 2 * n - 2, 2))


def test_matrix_chain_textbook_optimum():
    """Matrix-chain instance of Cormen et al., Introduction to Algorithms,
    Sec. 15.2: dims 30x35, 35x15, 15x5, 5x10, 10x20, 20x25; optimum 15125
    scalar multiplications with ((A1(A2A3))((A4A5)A6)).  Outer products are
    in the search space and must lose."""
    dims = [30, 35, 15, 5, 10, 20, 25]
    labs = "abcdefg"
    spec = ",".join(labs[i] + labs[i + 1] for i in range(6)) + "->ag"
    e = _e(spec, [(dims[i], dims[i + 1]) for i in range(6)])
    t, c, ties = O.optimal_tree(e, return_all=True)
    assert c == 15125
    assert t == ((0, (1, 2)), ((3, 4), 5))
    assert len(ties) == 1


def test_optimum_never_worse_than_any_tree():
    e = _e("bshw,rs,rt,rh,rw->bthw|hw", [(3, 5, 9, 7), (4, 5), (4, 6), (4, 3), (4, 2)])
    _, best = O.optimal_tree(e)
    costs = [O.tree_cost(e, t) for t in O.all_trees(range(5))]
    assert best == min(costs)


def test_canonical_tie_break_smallest_mask():
    """CP layer: convolving h before w or w before h costs the same; the
    canonical key takes the split whose first part has the smaller bitmask
    ({X,U_s,K_h} = 0b01011 before {X,U_s,K_w} = 0b10011)."""
    e = _e("bshw,rs,rt,rh,rw->bthw|hw", [(2, 16, 8, 8), (8, 16), (8, 16), (8, 3), (8, 3)])
    t, c, ties = O.optimal_tree(e, return_all=True)
    assert len(ties) == 2
    assert t == ((((0, 1), 3), 4), 2)
    assert ((((0, 1), 4), 3), 2) in ties
    # per-step costs: contract s, conv h (batch r), conv w, contract r
    B, S, T, R, H, W, K = 2, 16, 16, 8, 8, 8, 3
    assert O.step_costs(e, t) == [B * S * H * W * R, B * R * H * K * W, B * R * H * W * K,
                                  B * R * H * W * T]


def test_left_to_right_and_pairs():
    assert O.left_to_right_tree(4) == (((0, 1), 2), 3)
    from oracle.sequencer import tree_from_pairs
    # merged tensors go to the end of the list: left-to-right is (0,1),(0,2),(0,1)
    assert tree_from_pairs(4, [(0, 1), (0, 2), (0, 1)]) == (((0, 1), 2), 3)
    assert tree_from_pairs(4, [(0, 1), (0, 1), (0, 1)]) == ((0, 1), (2, 3))
    assert tree_from_pairs(4, [(1, 2), (0, 1), (0, 1)]) == ((0, 3), (1, 2))
    with pytest.raises(ValueError):
        tree_from_pairs(3, [(0, 1)])


def test_sequencer_example_figure1():
    """Figure 1 example (printed output missing from the paper).  Multi-way j
    is costed with the largest-size rule and the self-contracted m is summed
    before pairing; only optimality against every tree is checked, together
    with the value found by the survey's separate enumerator."""
    e = _e("ijk,jl,lmq,njpq->ijknp|j", [(4, 7, 9), (10, 5), (5, 4, 2), (6, 8, 9, 2)])
    t, c = O.optimal_tree(e)
    assert c == min(O.tree_cost(e, x) for x in O.all_trees(range(4)))
    assert (t, c) == ((0, ((1, 2), 3)), 144820)
    assert O.tree_cost(e, O.left_to_right_tree(4)) == 327240


def _chain_dp(p, cap):
    """Textbook matrix-chain interval DP (Cormen et al., Sec. 15.2) with every
    proper sub-chain product limited to `cap` elements (p[i] * p[j+1]);
    returns the least multiplication count, None when no parenthesisation fits."""
    n = len(p) - 1
    INF = float("inf")
    m = [[0 if i == j else INF for j in range(n)] for i in range(n)]
    for length in range(2, n + 1):
        for i in range(n - length + 1):
            j = i + length - 1
            if length < n and p[i] * p[j + 1] > cap:
                continue
            for k in range(i, j):
                c = m[i][k] + m[k + 1][j] + p[i] * p[k + 1] * p[j + 1]
                m[i][j] = min(m[i][j], c)
    return None if m[0][n - 1] == INF else m[0][n - 1]


@pytest.mark.parametrize("cap", [10 ** 9, 175, 174, 150, 125, 100, 90, 60])
def test_memory_limited_matrix_chain(cap):
    """The memory-limited search (Section 3.2, Figure 2) on the Cormen chain
    against an independent interval DP: same least cost under the cap (or
    both infeasible), and the returned tree respects the cap."""
    dims = [30, 35, 15, 5, 10, 20, 25]
    labs = "abcdefg"
    spec = ",".join(labs[i] + labs[i + 1] for i in range(6)) + "->ag"
    e = _e(spec, [(dims[i], dims[i + 1]) for i in range(6)])
    t, c = O.optimal_tree(e, max_elements=cap)
    ref = _chain_dp(dims, cap)
    if ref is None:
        assert t is None
    else:
        assert c == ref
        assert O.max_intermediate(e, t) <= cap
    if cap >= 175:   # the unconstrained optimum's largest intermediate is A2A3, 35 x 5
        assert t == ((0, (1, 2)), ((3, 4), 5))


def test_intermediate_size_matches_pairwise_evaluation():
    """intermediate_size equals the element count of the tensor the pairwise
    evaluator produces for that subset (a convolved label at its feature size)."""
    e = _e("bshw,rs,rt,rh,rw->bthw|hw", [(2, 5, 9, 7), (4, 5), (4, 6), (4, 3), (4, 2)])
    assert O.intermediate_size(e, (0, 1)) == 2 * 4 * 9 * 7      # Z1[b, r, h, w]
    assert O.intermediate_size(e, (1, 2)) == 4 * 5 * 6          # Us x Ut outer over r
    assert O.intermediate_size(e, (3, 4)) == 4 * 3 * 2          # Kh x Kw
    assert O.max_intermediate(e, ((((0, 1), 3), 4), 2)) == 2 * 4 * 9 * 7


def _chain_dp_step_cap(p, cap):
    """Matrix-chain interval DP (Cormen et al., Sec. 15.2) in which every
    multiplication of two sub-chain products may cost at most `cap`
    (p[i] * p[k+1] * p[j+1]); least total, None when nothing fits."""
    n = len(p) - 1
    INF = float("inf")
    m = [[0 if i == j else INF for j in range(n)] for i in range(n)]
    for length in range(2, n + 1):
        for i in range(n - length + 1):
            j = i + length - 1
            for k in range(i, j):
                step = p[i] * p[k + 1] * p[j + 1]
                if step <= cap:
                    m[i][j] = min(m[i][j], m[i][k] + m[k + 1][j] + step)
    return None if m[0][n - 1] == INF else m[0][n - 1]


@pytest.mark.parametrize("cap", [10 ** 9, 5250, 5249, 4500, 3750, 3000, 2625, 2000])
def test_cost_capped_matrix_chain(cap):
    """The per-node cost cap of Section 3.2, Figure 2 (the orange path) on the
    Cormen chain against an independent interval DP: same least total (or both
    infeasible), every step of the returned tree within the cap, and the
    unconstrained optimum whenever its largest step (A1 x (A2A3), 5250) fits."""
    dims = [30, 35, 15, 5, 10, 20, 25]
    labs = "abcdefg"
    spec = ",".join(labs[i] + labs[i + 1] for i in range(6)) + "->ag"
    e = _e(spec, [(dims[i], dims[i + 1]) for i in range(6)])
    t, c = O.optimal_tree(e, max_step_cost=cap)
    ref = _chain_dp_step_cap(dims, cap)
    if ref is None:
        assert t is None
    else:
        assert c == ref
        assert max(O.step_costs(e, t)) <= cap
    if cap >= 5250:
        assert t == ((0, (1, 2)), ((3, 4), 5)) and c == 15125
    else:
        assert ref is None or ref > 15125


@pytest.mark.parametrize("name", ["rtt_conv", "tr_conv", "cp_conv"])
def test_cost_cap_on_layer_strings(name):
    """Layer strings of Appendix A.3: with a cap one below the optimum's
    largest step, the capped search returns the cheapest tree whose every step
    fits, checked against every tree; where no tree has a smaller largest step
    (the CP layer: some step always contracts X with U_s), it returns none."""
    import conftest
    spec = conftest.load_layer_strings()[name][0]
    shapes = conftest.PAPER_SHAPES[name]
    e = _e(spec, shapes)
    t0, c0 = O.optimal_tree(e)
    big = max(O.step_costs(e, t0))
    t1, c1 = O.optimal_tree(e, max_step_cost=big - 1)
    fits = [x for x in O.all_trees(range(e.n)) if max(O.step_costs(e, x)) <= big - 1]
    if not fits:
        assert (t1, c1) == (None, None)
        return
    assert c1 == min(O.tree_cost(e, x) for x in fits) and c1 > c0
    assert max(O.step_costs(e, t1)) <= big - 1
    assert O.optimal_tree(e, max_step_cost=big) == (t0, c0)


def test_checkpoint_choice_hand_values():
    """Keep-or-recompute choice on the tiny CP layer (Section 3.3), hand
    values: the planned tree's intermediates are Z1 = X*Us, Z2 = Z1 conv Kh,
    Z3 = Z2 conv Kw, each [b=2, r=8, 8, 8] = 1024 elements (4096 B in fp32),
    spared recompute costs 16384, 3072 and 3072 multiplications."""
    e = _e("bshw,rs,rt,rh,rw->bthw|hw", [(2, 16, 8, 8), (8, 16), (8, 16), (8, 3), (8, 3)])
    t = O.optimal_tree(e)[0]
    assert O.checkpoint_choice(e, t, 0, 4) == (set(), 0, 16384 + 3072 + 3072)
    assert O.checkpoint_choice(e, t, 4095, 4) == (set(), 0, 22528)
    assert O.checkpoint_choice(e, t, 4096, 4) == ({0}, 4096, 6144)
    # two fit: Z1 and the lower-indexed of the two equal conv results
    assert O.checkpoint_choice(e, t, 8192 + 100, 4) == ({0, 1}, 8192, 3072)
    assert O.checkpoint_choice(e, t, 10 ** 9, 4) == ({0, 1, 2}, 12288, 0)
    # bf16 halves the bytes
    assert O.checkpoint_choice(e, t, 4096, 2) == ({0, 1}, 4096, 3072)


def test_checkpoint_choice_is_the_best_subset():
    """Against a direct scan of every subset of the tensor-train layer's
    intermediates: no subset within the budget spares more."""
    import conftest
    spec = conftest.load_layer_strings()["rtt_conv"][0]
    e = _e(spec, conftest.PAPER_SHAPES["rtt_conv"])
    t = O.optimal_tree(e)[0]
    steps = O.post_order_steps(t)[:-1]
    sizes = [O.intermediate_size(e, O.leaves(a) + O.leaves(b)) * 4 for a, b in steps]
    costs = [O.step_cost(e, O.leaves(a), O.leaves(b)) for a, b in steps]
    for budget in [0, min(sizes), sum(sizes) // 2, sum(sizes) - 1, sum(sizes)]:
        kept, w, rest = O.checkpoint_choice(e, t, budget, 4)
        assert w <= budget and w == sum(sizes[s] for s in kept)
        assert rest == sum(costs) - sum(costs[s] for s in kept)
        best = max(sum(c for c, k in zip(costs, m) if k)
                   for m in itertools.product([0, 1], repeat=len(steps))
                   if sum(s for s, k in zip(sizes, m) if k) <= budget)
        assert sum(costs) - rest == best
