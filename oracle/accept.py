"""fp64 oracle of speculative acceptance and the final sample (test infrastructure).

Notation: p is the TARGET model's distribution, q the DRAFT (small
speculative model's) distribution.  The paper's Eq. (1) uses the opposite
letters (its p is the SSM's, its q the LLM's) and accepts a candidate with
probability min(1, target/draft); only the letters differ.

Chain (Sec. 2.2, Eq. (1); Sec. 4.3 for the extra token), per request with k
drafts x_1..x_k and k+1 target rows:

  p_j = softmax(target_logits[row j])              j = 0..k   (row j scores x_{j+1})
  q_j = draft_probs[row j] as stored               j = 0..k-1
  draft j is accepted iff u_j * q_j(x) < p_j(x)    (= u_j < min(1, p/q) for q > 0, u < 1)
  a = index of the first rejection, or k if none
  w = max(0, p_a - q_a) if a < k  (residual distribution, Sec. 2.2)
      p_k               if a = k  (the LLM's one additional token, Sec. 4.3)
      p_a               if a < k and sum(w) == 0 (only reachable through rounding)
  next = smallest v with sum_{t<=v} w_t > u_k * sum(w)   (inverse CDF, ids ascending)

Tree (token-tree verification as in SpecInfer, cited in Sec. 5.1 and Sec. 6.1;
the paper does not spell the rule out), read as: node n >= 1 is accepted iff
its parent is accepted and u_{n-1} * q_par(x_n) < p_par(x_n), where par is
its parent's target row and draft row; n* = the deepest accepted node,
smallest BFS index on ties; accepted length = depth(n*); the final token is
drawn from p_{n*} if n* is a leaf, else from max(0, p_{n*} - q_{n*}) (same
zero-mass fallback).  For a path-shaped tree this is exactly the chain.

Near ties.  An implementation in finite precision can legitimately differ
from these fp64 results only near a decision boundary, so two distances are
reported for every request:
  * acceptance tests on the decision path: |u_j - min(1, p/q)|, a tie below
    NEAR_TIE = 1e-5;
  * the final sample: the distance, in probability mass, between the target
    u * sum(w) and the cumulative weights that bracket the chosen token, a tie
    below NEAR_TIE_MASS = 2e-7.  (A sampler whose sums are exact to ~1e-8 of
    probability mass -- fp64 accumulation over fp32 entries -- can only pick
    a different token inside this band.)
"""
from __future__ import annotations

from typing import Optional, Sequence

import numpy as np

from .attention import widen

NEAR_TIE = 1e-5
NEAR_TIE_MASS = 2e-7


def softmax64(logits: np.ndarray) -> np.ndarray:
    """Target distribution of one row (fp64, max-subtracted)."""
    x = np.asarray(logits, dtype=np.float64)
    e = np.exp(x - x.max())
    return e / e.sum()


def inverse_cdf(w: np.ndarray, u: float):
    """Smallest v with cumsum(w)[v] > u * sum(w), and the distance (in the
    units of w) from u * sum(w) to the cumulative weights bracketing v.

    Zero-weight tokens are never chosen; a target that rounds past the total
    is clamped to the last token with positive weight.
    """
    w = np.asarray(w, dtype=np.float64)
    cdf = np.cumsum(w)
    target = u * cdf[-1]
    v = int(np.searchsorted(cdf, target, side="right"))
    # cdf[v] > target >= cdf[v-1] forces w[v] > 0; only an overshoot needs a clamp
    if v >= len(w):
        v = int(np.nonzero(w > 0)[0][-1])
    c_lo = cdf[v - 1] if v > 0 else 0.0
    margin = min(abs(target - c_lo), abs(cdf[v] - target))
    return v, margin


def _test(u: float, px: float, qx: float):
    """Acceptance test u*q(x) < p(x) and its distance to the boundary."""
    accept = u * qx < px
    if qx > 0:
        margin = abs(u - min(1.0, px / qx))
    else:
        margin = np.inf
    return bool(accept), margin


def _result(length, nxt, node, test_margins, sample_margin) -> dict:
    mt = float(min(test_margins)) if test_margins else np.inf
    return {"accepted_len": length, "next_token": nxt, "accepted_node": node,
            "margin": mt, "margin_mass": float(sample_margin),
            "near_tie": bool(mt < NEAR_TIE or sample_margin < NEAR_TIE_MASS)}


def accept_chain(p_rows: np.ndarray, q_rows: np.ndarray, tokens: Sequence[int],
                 uniforms: Sequence[float]) -> dict:
    """One request of the chain rule.  p_rows [k+1, V] (target probabilities),
    q_rows [k, V] (draft probabilities), tokens [k], uniforms [k+1]."""
    k = len(tokens)
    margins = []
    a = k
    for j in range(k):
        x = int(tokens[j])
        ok, m = _test(float(uniforms[j]), p_rows[j, x], q_rows[j, x])
        margins.append(m)
        if not ok:
            a = j
            break
    if a < k:
        w = np.maximum(0.0, p_rows[a] - q_rows[a])
        if w.sum() <= 0.0:
            w = p_rows[a]
    else:
        w = p_rows[k]
    nxt, m_s = inverse_cdf(w, float(uniforms[k]))
    return _result(a, nxt, a, margins, m_s)


def tree_depths(parent: Sequence[int]) -> np.ndarray:
    depth = np.zeros(len(parent), dtype=np.int64)
    for n in range(1, len(parent)):
        depth[n] = depth[int(parent[n])] + 1
    return depth


def accept_tree_sequential(p_rows: np.ndarray, q_rows: dict, tokens: Sequence[int],
                           uniforms: Sequence[float], parent: Sequence[int]) -> dict:
    """One request of sequential sibling verification over a token tree, the
    multi-step speculative sampling of SpecInfer (the token-tree system the
    paper's evaluation follows, Sec. 5.1).  Starting at the root, the current
    node's children -- drafted i.i.d. from its draft row q -- are tested in
    BFS order against a running target distribution p' (first the node's own
    target row): child c is accepted iff u_c * q(x_c) < p'(x_c); a rejection
    replaces p' by max(0, p' - q) normalised (kept as it is if that has zero
    mass, reachable only through rounding).  The first accepted child becomes
    the current node; when no child is accepted, or the node is a leaf, the
    final token is drawn from p' with the last uniform.  Arguments as for
    accept_tree."""
    n = len(parent)
    depth = tree_depths(parent)
    children = {u: [c for c in range(1, n) if int(parent[c]) == u] for u in range(n)}
    node, margins = 0, []
    while True:
        pp = np.asarray(p_rows[node], dtype=np.float64)
        nxt_node = None
        for c in children[node]:
            q = q_rows[node]
            x = int(tokens[c - 1])
            ok, m = _test(float(uniforms[c - 1]), pp[x], q[x])
            margins.append(m)
            if ok:
                nxt_node = c
                break
            w = np.maximum(0.0, pp - q)
            if w.sum() > 0.0:
                pp = w / w.sum()
        if nxt_node is None:
            break
        node = nxt_node
    nxt, m_s = inverse_cdf(pp, float(uniforms[n - 1]))
    return _result(int(depth[node]), nxt, node, margins, m_s)


def accept_tree(p_rows: np.ndarray, q_rows: dict, tokens: Sequence[int],
                uniforms: Sequence[float], parent: Sequence[int]) -> dict:
    """One request of the tree rule.  p_rows [n, V]; q_rows maps each node that
    has children to its draft row; tokens[n-1] is node n's token; uniforms [n]."""
    n = len(parent)
    depth = tree_depths(parent)
    has_child = set(int(x) for x in parent[1:])
    accepted = np.zeros(n, dtype=bool)
    accepted[0] = True
    margins = []
    for node in range(1, n):
        par = int(parent[node])
        if not accepted[par]:
            continue
        x = int(tokens[node - 1])
        ok, m = _test(float(uniforms[node - 1]), p_rows[par, x], q_rows[par][x])
        margins.append(m)
        accepted[node] = ok
    best = 0
    for node in range(1, n):
        if accepted[node] and depth[node] > depth[best]:
            best = node
    if best in has_child:
        w = np.maximum(0.0, p_rows[best] - q_rows[best])
        if w.sum() <= 0.0:
            w = p_rows[best]
    else:
        w = p_rows[best]
    nxt, m_s = inverse_cdf(w, float(uniforms[n - 1]))
    return _result(int(depth[best]), nxt, best, margins, m_s)


def verify_accept(target_logits: np.ndarray, draft_probs: np.ndarray,
                  draft_tokens: np.ndarray, uniforms: np.ndarray,
                  n_q: Sequence[int], dtype: str = "f32",
                  tree_parent: Optional[Sequence[int]] = None,
                  requests: Optional[Sequence[int]] = None,
                  tree_rule: str = "independent",
                  tree_parents: Optional[Sequence[Sequence[int]]] = None) -> dict:
    """Acceptance for a packed batch (layouts as in the C interface).

    Request i owns target rows q0_i .. q0_i + n_i - 1 (q0 = running sum of
    n_i), uniforms at the same rows, draft tokens q0_i - i .. q0_i - i + n_i - 2
    (one per non-root node) and draft rows d0_i .. (d0 = running sum of the
    number of nodes with children: k_i for a chain).  A token tree is shared
    (tree_parent) or given per request (tree_parents[i]).  ``requests``
    restricts the work to a subset (results for the others are -1).
    """
    n_q = [int(x) for x in n_q]
    B = len(n_q)
    pars = [tree_parents[i] if tree_parents is not None else tree_parent for i in range(B)]
    inner = [None if par is None else sorted(set(int(x) for x in par[1:])) for par in pars]
    n_int = [n - 1 if inner[i] is None else len(inner[i]) for i, n in enumerate(n_q)]
    q0 = np.concatenate([[0], np.cumsum(n_q)]).astype(np.int64)
    d0 = np.concatenate([[0], np.cumsum(n_int)]).astype(np.int64)
    keys = ("accepted_len", "next_token", "accepted_node")
    res = {key: np.full(B, -1, dtype=np.int64) for key in keys}
    res["near_tie"] = np.zeros(B, dtype=bool)
    res["margin"] = np.full(B, np.inf)
    res["margin_mass"] = np.full(B, np.inf)
    todo = range(B) if requests is None else requests
    for i in todo:
        n = n_q[i]
        p_rows = np.stack([softmax64(widen(target_logits[q0[i] + j], dtype)) for j in range(n)])
        toks = np.asarray(draft_tokens[q0[i] - i: q0[i] - i + n - 1], dtype=np.int64)
        us = np.asarray(uniforms[q0[i]: q0[i] + n], dtype=np.float64)
        if pars[i] is None:
            q_rows = widen(draft_probs[d0[i]: d0[i] + n - 1], dtype).reshape(n - 1, target_logits.shape[1])
            r = accept_chain(p_rows, q_rows, toks, us)
        else:
            if len(pars[i]) != n:
                raise ValueError("tree size must equal the number of verify nodes")
            q_rows = {node: widen(draft_probs[d0[i] + rnk], dtype) for rnk, node in enumerate(inner[i])}
            rule = accept_tree_sequential if tree_rule == "sequential" else accept_tree
            r = rule(p_rows, q_rows, toks, us, pars[i])
        for key in keys:
            res[key][i] = r[key]
        res["near_tie"][i] = r["near_tie"]
        res["margin"][i] = r["margin"]
        res["margin_mass"][i] = r["margin_mass"]
    return res
