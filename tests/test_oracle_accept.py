"""Pins of the fp64 acceptance oracle against facts outside itself.

The main pin is the defining property of speculative sampling (Eq. (1) with
the residual resample of Sec. 2.2): the token a round emits is distributed
exactly as the target distribution.  The oracle is a deterministic function
of its uniforms, piecewise constant between known breakpoints, so the
probability of every outcome is computed EXACTLY by enumerating uniform cells
(no Monte Carlo) and must equal the target probabilities to 1e-12.  Closed
forms for the accepted-length distribution and special cases complete it.
"""
import itertools

import numpy as np
import pytest

from oracle import accept_chain, accept_tree, verify_accept, softmax64, inverse_cdf

RNG = np.random.default_rng(99)


def _dist(V, rng=RNG, zeros=0):
    p = rng.random(V) ** 2 + 1e-3
    if zeros:
        p[rng.choice(V, zeros, replace=False)] = 0.0
    return p / p.sum()


def _cells(breaks):
    """Cells of [0, 1) cut at the given breakpoints -> (midpoint, length)."""
    b = sorted(set([0.0, 1.0] + [float(x) for x in breaks if 0.0 < x < 1.0]))
    return [((lo + hi) / 2.0, hi - lo) for lo, hi in zip(b[:-1], b[1:])]


def _cdf_breaks(*ws):
    out = []
    for w in ws:
        w = np.asarray(w, np.float64)
        if w.sum() > 0:
            out.extend(np.cumsum(w) / w.sum())
    return out


def _ratio(p, q, x):
    return min(1.0, p[x] / q[x])


def _first_token_distribution(p0, q0, p1):
    V = len(p0)
    dist = np.zeros(V)
    fin = _cdf_breaks(np.maximum(0, p0 - q0), p0, p1)
    for x in range(V):
        if q0[x] == 0:
            continue
        for u0, l0 in _cells([_ratio(p0, q0, x)]):
            for u1, l1 in _cells(fin):
                r = accept_chain(np.stack([p0, p1]), q0[None], [x], [u0, u1])
                y = x if r["accepted_len"] == 1 else r["next_token"]
                dist[y] += q0[x] * l0 * l1
    return dist


def _edge_rows(V):
    p = _dist(V)
    yield "random", p, _dist(V)
    yield "p_equals_q", p, p.copy()
    a = np.zeros(V); a[:V // 2] = _dist(V // 2)
    b = np.zeros(V); b[V // 2:] = _dist(V - V // 2)
    yield "disjoint", a, b
    oh = np.zeros(V); oh[3] = 1.0
    yield "onehot_q", p, oh
    yield "p_with_zeros", _dist(V, zeros=3), _dist(V)
    yield "q_with_zeros", _dist(V), _dist(V, zeros=3)


@pytest.mark.parametrize("case", range(6))
def test_emitted_token_is_distributed_as_target(case):
    name, p0, q0 = list(_edge_rows(8))[case]
    p1 = _dist(8)
    dist = _first_token_distribution(p0, q0, p1)
    np.testing.assert_allclose(dist, p0, rtol=0, atol=1e-12, err_msg=name)


@pytest.mark.parametrize("trial", range(3))
def test_random_rows_identity(trial):
    rng = np.random.default_rng(1000 + trial)
    p0, q0, p1 = _dist(8, rng), _dist(8, rng), _dist(8, rng)
    np.testing.assert_allclose(_first_token_distribution(p0, q0, p1), p0, rtol=0, atol=1e-12)


def test_two_token_identity_with_prefix_dependent_rows():
    """k = 2: the first two emitted tokens follow p(y1) p(y2 | y1).

    Target and draft rows after the first draft depend on that draft.  If the
    round emits only one token, the next round starts from it and (by the
    one-token identity) emits p(. | y1).
    """
    V = 8
    rng = np.random.default_rng(7)
    p0, q0 = _dist(V, rng), _dist(V, rng)
    p1 = {x: _dist(V, rng) for x in range(V)}            # p(. | x1)
    q1 = {x: _dist(V, rng) for x in range(V)}
    p2 = {(x, y): _dist(V, rng) for x in range(V) for y in range(V)}
    joint = np.zeros((V, V))
    for x1 in range(V):
        for u0, l0 in _cells([_ratio(p0, q0, x1)]):
            for x2 in range(V):
                for u1, l1 in _cells([_ratio(p1[x1], q1[x1], x2)]):
                    fin = _cdf_breaks(np.maximum(0, p0 - q0), np.maximum(0, p1[x1] - q1[x1]), p2[(x1, x2)],
                                      p0, p1[x1])
                    for u2, l2 in _cells(fin):
                        w = q0[x1] * l0 * q1[x1][x2] * l1 * l2
                        r = accept_chain(np.stack([p0, p1[x1], p2[(x1, x2)]]), np.stack([q0, q1[x1]]),
                                         [x1, x2], [u0, u1, u2])
                        a, nxt = r["accepted_len"], r["next_token"]
                        if a == 0:
                            joint[nxt] += w * p1[nxt]             # second token from the next round
                        elif a == 1:
                            joint[x1, nxt] += w
                        else:
                            joint[x1, x2] += w
    expect = p0[:, None] * np.stack([p1[y] for y in range(V)])
    np.testing.assert_allclose(joint, expect, rtol=0, atol=1e-12)


def test_accepted_length_distribution_closed_form():
    """Rows independent of the prefix: P(a >= j) = prod_{t<j} sum_x min(p_t, q_t)."""
    V, k = 8, 3
    rng = np.random.default_rng(11)
    P = [_dist(V, rng) for _ in range(k + 1)]
    Q = [_dist(V, rng) for _ in range(k)]
    alpha = [np.minimum(P[t], Q[t]).sum() for t in range(k)]
    pa = np.zeros(k + 1)
    for xs in itertools.product(range(V), repeat=k):
        for cells in itertools.product(*[_cells([_ratio(P[t], Q[t], xs[t])]) for t in range(k)]):
            w = np.prod([Q[t][xs[t]] for t in range(k)]) * np.prod([c[1] for c in cells])
            r = accept_chain(np.stack(P), np.stack(Q), list(xs), [c[0] for c in cells] + [0.5])
            pa[r["accepted_len"]] += w
    tail = [np.prod(alpha[:j]) for j in range(k + 2)]
    expect = np.array([tail[j] - tail[j + 1] for j in range(k)] + [tail[k]])
    np.testing.assert_allclose(pa, expect, rtol=0, atol=1e-12)
    # mean accepted = sum_j prod_{t<j} alpha_t  (the n*A accepted drafts per round)
    assert abs((pa * np.arange(k + 1)).sum() - sum(tail[1:k + 1])) < 1e-12


def test_softmax_closed_form():
    p = _dist(16)
    np.testing.assert_allclose(softmax64(np.log(p) + 3.7), p, rtol=1e-13)
    np.testing.assert_allclose(softmax64(np.array([0.0, np.log(3.0)])), [0.25, 0.75], rtol=1e-15)


def test_inverse_cdf_convention():
    w = np.array([0.125, 0.0, 0.25, 0.25, 0.375])
    # cumulative 0.125 0.125 0.375 0.625 1.0 (exact): smallest v with cumulative > u
    assert inverse_cdf(w, 0.0)[0] == 0
    assert inverse_cdf(w, 0.125)[0] == 2        # boundary goes up; zero-weight id 1 skipped
    assert inverse_cdf(w, 0.25)[0] == 2
    assert inverse_cdf(w, 0.375)[0] == 3
    assert inverse_cdf(w, 0.999)[0] == 4
    assert inverse_cdf(np.array([0.0, 0.0, 2.0, 0.0]), 0.7)[0] == 2   # unnormalised weights
    assert inverse_cdf(np.array([0.0, 5.0, 0.0]), 0.0)[0] == 1


def test_special_cases():
    V = 8
    p = _dist(V, zeros=2)
    zero_tok = int(np.nonzero(p == 0)[0][0])
    pos_tok = int(np.nonzero(p > 0)[0][0])
    q = _dist(V)
    # u = 0 accepts iff p(x) > 0
    assert accept_chain(np.stack([p, p]), q[None], [pos_tok], [0.0, 0.5])["accepted_len"] == 1
    assert accept_chain(np.stack([p, p]), q[None], [zero_tok], [0.0, 0.5])["accepted_len"] == 0
    # p == q accepts every draft, for any uniform below 1
    rows = np.stack([_dist(V) for _ in range(4)])
    for u in (0.0, 0.5, 1 - 2 ** -24):
        assert accept_chain(rows, rows[:3], [1, 2, 3], [u] * 4)["accepted_len"] == 3
    # one-hot draft on a token the target never emits: reject, resample from p itself
    oh = np.zeros(V); oh[zero_tok] = 1.0
    r = accept_chain(np.stack([p, p]), oh[None], [zero_tok], [0.3, 0.6])
    assert r["accepted_len"] == 0
    assert r["next_token"] == inverse_cdf(p, 0.6)[0]
    # k = 0 is plain sampling from the single target row
    p4 = np.array([0.1, 0.2, 0.3, 0.4])
    assert accept_chain(p4[None], np.zeros((0, 4)), [], [0.25])["next_token"] == 1
    assert accept_chain(p4[None], np.zeros((0, 4)), [], [0.65])["next_token"] == 3
    # a residual with one positive entry returns that token whatever the uniform
    p1 = np.array([0.5, 0.5, 0.0, 0.0]); q1 = np.array([0.5, 0.25, 0.25, 0.0])
    for u in (0.0, 0.4, 0.99):
        r = accept_chain(np.stack([p1, p4]), q1[None], [2], [0.1, u])
        assert (r["accepted_len"], r["next_token"]) == (0, 1)
    # zero residual mass (draft row scaled above the target): fall back to p_a
    qs = 1.1 * p4
    r = accept_chain(np.stack([p4, p4]), qs[None], [3], [0.95, 0.65])
    assert r["accepted_len"] == 0 and r["next_token"] == 3


def test_accepted_length_bounds_random_batches():
    rng = np.random.default_rng(5)
    for _ in range(50):
        k = int(rng.integers(0, 6))
        P = np.stack([_dist(16, rng) for _ in range(k + 1)])
        Q = np.stack([_dist(16, rng) for _ in range(k)]) if k else np.zeros((0, 16))
        toks = rng.integers(0, 16, size=k)
        r = accept_chain(P, Q, toks, rng.random(k + 1))
        assert 0 <= r["accepted_len"] <= k
        assert 0 <= r["next_token"] < 16


def test_batch_packing_by_hand():
    """The packed batch layout (target rows and uniforms at q0_i, draft tokens
    at q0_i - i, draft rows at d0_i) against a two-request case worked by
    hand: a swapped or shifted index changes an output."""
    from parity_util import hand_packed_case
    inp, expect = hand_packed_case()
    r = verify_accept(inp["target_logits"], inp["draft_probs"], inp["draft_tokens"], inp["uniforms"],
                      inp["draft_len"] + 1)
    assert r["accepted_len"].tolist() == expect["accepted_len"]
    assert r["next_token"].tolist() == expect["next_token"]
    assert not r["near_tie"].any()


@pytest.mark.parametrize("rule", ["independent", "sequential"])
def test_per_request_trees_by_hand(rule):
    """Per-request topologies: the packing (target rows and uniforms at q0_i,
    node tokens at q0_i - i, draft rows at d0_i = running count of nodes with
    children) against a two-request case worked by hand under each rule."""
    from parity_util import hand_packed_trees
    inp, expect = hand_packed_trees()
    r = verify_accept(inp["target_logits"], inp["draft_probs"], inp["draft_tokens"], inp["uniforms"],
                      [len(x) for x in inp["parents"]], tree_parents=inp["parents"], tree_rule=rule)
    for key, val in expect[rule].items():
        assert r[key].tolist() == val, (rule, key, r[key])
    assert not r["near_tie"].any()


@pytest.mark.parametrize("rule", ["independent", "sequential"])
def test_per_request_paths_and_shared_trees(rule):
    """Per-request trees that are all paths decide exactly as chains; per-request
    trees that are all equal decide exactly as the shared tree."""
    rng = np.random.default_rng(8)
    V = 32
    n_q = [4, 1, 6, 3]
    logits = rng.standard_normal((sum(n_q), V)).astype(np.float32)
    probs = np.stack([_dist(V, rng) for _ in range(sum(n_q) - len(n_q))]).astype(np.float32)
    toks = rng.integers(0, V, size=sum(n_q) - len(n_q)).astype(np.int32)
    us = rng.random(sum(n_q)).astype(np.float32)
    chain = verify_accept(logits, probs, toks, us, n_q)
    paths = verify_accept(logits, probs, toks, us, n_q, tree_parents=[list(range(-1, n - 1)) for n in n_q],
                          tree_rule=rule)
    for key in ("accepted_len", "next_token", "accepted_node", "near_tie"):
        np.testing.assert_array_equal(chain[key], paths[key])
    tree = [-1, 0, 0, 1, 1, 2]
    B = 5
    logits = rng.standard_normal((6 * B, V)).astype(np.float32)
    probs = np.stack([_dist(V, rng) for _ in range(3 * B)]).astype(np.float32)
    toks = rng.integers(0, V, size=5 * B).astype(np.int32)
    us = rng.random(6 * B).astype(np.float32)
    shared = verify_accept(logits, probs, toks, us, [6] * B, tree_parent=tree, tree_rule=rule)
    per = verify_accept(logits, probs, toks, us, [6] * B, tree_parents=[tree] * B, tree_rule=rule)
    for key in ("accepted_len", "next_token", "accepted_node", "near_tie"):
        np.testing.assert_array_equal(shared[key], per[key])


# ------------------------------------------------------------------- trees
def test_path_tree_equals_chain_batch():
    rng = np.random.default_rng(3)
    B, n, V = 5, 5, 32
    logits = rng.standard_normal((B * n, V)).astype(np.float32)
    probs = np.stack([_dist(V, rng) for _ in range(B * (n - 1))]).astype(np.float32)
    toks = rng.integers(0, V, size=B * (n - 1)).astype(np.int32)
    us = rng.random(B * n).astype(np.float32)
    chain = verify_accept(logits, probs, toks, us, [n] * B)
    path = verify_accept(logits, probs, toks, us, [n] * B, tree_parent=[-1, 0, 1, 2, 3])
    for key in ("accepted_len", "next_token", "accepted_node", "near_tie"):
        np.testing.assert_array_equal(chain[key], path[key])


def test_three_node_tree_distribution_reading():
    """Root with two leaf children, both drafted from the root's q.

    Under the per-node rule: node 1 wins when accepted; else node 2 when
    accepted; else the root with a residual sample.  Closed form:
    P(n*=1, z) = a p1(z), P(n*=2, z) = (1-a) a p2(z), P(n*=0, z) = (1-a)^2 r(z)
    with a = sum min(p0, q0) and r the normalised residual.
    """
    V = 4
    rng = np.random.default_rng(21)
    p0, p1, p2, q0 = _dist(V, rng), _dist(V, rng), _dist(V, rng), _dist(V, rng)
    parent = [-1, 0, 0]
    res = np.maximum(0, p0 - q0)
    got = np.zeros((3, V))
    fin = _cdf_breaks(res, p1, p2)
    for x1 in range(V):
        for x2 in range(V):
            for (u1, l1), (u2, l2) in itertools.product(_cells([_ratio(p0, q0, x1)]), _cells([_ratio(p0, q0, x2)])):
                for u3, l3 in _cells(fin):
                    r = accept_tree(np.stack([p0, p1, p2]), {0: q0}, [x1, x2], [u1, u2, u3], parent)
                    got[r["accepted_node"], r["next_token"]] += q0[x1] * q0[x2] * l1 * l2 * l3
                    assert r["accepted_len"] == (0 if r["accepted_node"] == 0 else 1)
    a = np.minimum(p0, q0).sum()
    expect = np.stack([(1 - a) ** 2 * res / res.sum(), a * p1, (1 - a) * a * p2])
    np.testing.assert_allclose(got, expect, rtol=0, atol=1e-12)


def test_tree_deepest_node_smallest_index():
    V = 8
    parent = [-1, 0, 0, 1, 1, 2, 2]
    P = np.stack([_dist(V) for _ in range(7)])
    Q = {n: _dist(V) for n in (0, 1, 2)}
    toks = [0, 1, 2, 3, 4, 5]
    r = accept_tree(P, Q, toks, [0.0] * 6 + [0.5], parent)      # every test passes (p > 0)
    assert (r["accepted_node"], r["accepted_len"]) == (3, 2)
    assert r["next_token"] == inverse_cdf(P[3], 0.5)[0]
    # reject node 1 (u just below 1 and p/q < 1): the depth-2 winner moves under node 2
    toks2 = [int(np.argmin(P[0] / Q[0])), 1, 2, 3, 4, 5]
    r = accept_tree(P, Q, toks2, [1 - 2 ** -24] + [0.0] * 5 + [0.5], parent)
    assert (r["accepted_node"], r["accepted_len"]) == (5, 2)


def _sibling_first_token(p0, q0, child_rows, m):
    """Distribution of the first emitted token of a one-level tree with m
    children drafted i.i.d. from q0, by enumerating the child tokens and the
    cells of every uniform (cut where a decision can change)."""
    from oracle import accept_tree_sequential
    V = len(p0)
    parent = [-1] + [0] * m
    p_rows = np.stack([p0] + child_rows)
    # the running distributions after 0..m rejections do not depend on the tokens
    runs = [p0]
    for _ in range(m):
        w = np.maximum(0.0, runs[-1] - q0)
        runs.append(w / w.sum() if w.sum() > 0 else runs[-1])
    dist = np.zeros(V)
    for xs in itertools.product(range(V), repeat=m):
        wq = np.prod([q0[x] for x in xs])
        if wq == 0:
            continue
        test_cells = [_cells([min(1.0, runs[i][x] / q0[x])]) for i, x in enumerate(xs)]
        for combo in itertools.product(*test_cells):
            us = [c[0] for c in combo]
            lw = np.prod([c[1] for c in combo])
            for uf, lf in _cells(_cdf_breaks(runs[m])):
                r = accept_tree_sequential(p_rows, {0: q0}, list(xs), us + [uf], parent)
                y = list(xs)[r["accepted_node"] - 1] if r["accepted_len"] == 1 else r["next_token"]
                dist[y] += wq * lw * lf
    return dist


@pytest.mark.parametrize("m", [2, 3])
@pytest.mark.parametrize("case", range(4))
def test_sequential_siblings_preserve_the_target(m, case):
    """SpecInfer's guarantee: with children drafted i.i.d. from q, sequential
    sibling verification emits a first token distributed exactly as p."""
    V = 8
    rng = np.random.default_rng(50 + case)
    if case == 0:
        p0, q0 = _dist(V, rng), _dist(V, rng)
    elif case == 1:                                   # p = q: the first child is always accepted
        p0 = _dist(V, rng)
        q0 = p0.copy()
    elif case == 2:                                   # disjoint supports: every child rejected
        p0 = np.r_[_dist(4, rng), np.zeros(4)]
        q0 = np.r_[np.zeros(4), _dist(4, rng)]
    else:                                             # one-hot draft
        p0, q0 = _dist(V, rng), np.eye(V)[3]
    child_rows = [_dist(V, rng) for _ in range(m)]
    np.testing.assert_allclose(_sibling_first_token(p0, q0, child_rows, m), p0, rtol=0, atol=1e-12)


def test_sequential_on_a_path_is_the_chain_rule():
    """Every node with one child: sequential sibling verification is the chain
    rule, decision for decision."""
    from oracle import accept_tree_sequential
    rng = np.random.default_rng(9)
    V, k = 16, 4
    for _ in range(200):
        p_rows = np.stack([_dist(V, rng) for _ in range(k + 1)])
        q_rows = np.stack([_dist(V, rng) for _ in range(k)])
        toks = [int(rng.integers(V)) for _ in range(k)]
        us = list(rng.random(k + 1))
        a = accept_chain(p_rows, q_rows, toks, us)
        b = accept_tree_sequential(p_rows, {j: q_rows[j] for j in range(k)}, toks, us, [-1, 0, 1, 2, 3])
        assert (a["accepted_len"], a["next_token"]) == (b["accepted_len"], b["next_token"])


def test_sequential_siblings_by_hand():
    """p = (.5, .3, .2), q = (.2, .5, .3), both children draft token 1.  Child
    1: u = .7, .7 * .5 = .35 >= .3, rejected; p' = norm(max(0, p - q)) =
    (1, 0, 0).  Child 2: p'(1) = 0, rejected; p'' = norm(max(0, p' - q)) =
    (1, 0, 0).  The final token is 0, at the root."""
    from oracle import accept_tree_sequential
    p0, q0 = np.array([0.5, 0.3, 0.2]), np.array([0.2, 0.5, 0.3])
    rows = np.stack([p0, p0, p0])
    r = accept_tree_sequential(rows, {0: q0}, [1, 1], [0.7, 0.1, 0.5], [-1, 0, 0])
    assert (r["accepted_len"], r["accepted_node"], r["next_token"]) == (0, 0, 0)
    # u = .5 accepts child 1 (.25 < .3): the bonus comes from row 1
    rows2 = np.stack([p0, np.array([0.0, 0.0, 1.0]), p0])
    r = accept_tree_sequential(rows2, {0: q0}, [1, 1], [0.5, 0.1, 0.5], [-1, 0, 0])
    assert (r["accepted_len"], r["accepted_node"], r["next_token"]) == (1, 1, 2)
