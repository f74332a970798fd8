"""fp64 oracle of verify attention (test infrastructure; see package header).

Definition followed (paper Sec. 2.1 for the KV cache, Sec. 2.2 for verifying
all candidate tokens in one parallel forward of the target model; the
attention formula itself is the standard scaled dot-product softmax
attention, which the paper uses without writing out):

For request i with c_i cached positions and n_i verify nodes (the last
accepted token plus the drafts; for a token tree, its nodes in BFS order),
query head h and verify node j:

    g      = h // (Hq / Hkv)                       (grouped-query head map)
    A(i,j) = {0 .. c_i-1} U {c_i + t : t in anc*(j)}
    s_t    = scale * <Q[q0_i + j, h, :], K[kv0_i + t, g, :]>     for t in A(i,j)
    w      = softmax(s)
    O[q0_i + j, h, :] = sum_t w_t V[kv0_i + t, g, :]

anc*(j) is the set of ancestors of node j together with j itself: {0..j} for
a chain (causal mask inside the verify block), the root-to-node path for a
tree.  A token tree is either shared by every request of the batch or given
per request (each request its own BFS parent array).  The verify block's keys
and values are the last n_i rows of the request's KV rows.  scale defaults to
1/sqrt(d).
"""
from __future__ import annotations

from typing import Optional, Sequence

import numpy as np


def widen(x: np.ndarray, dtype: str) -> np.ndarray:
    """Stored values -> float64.  bf16 is held as raw uint16 bit patterns."""
    if dtype == "bf16":
        bits = np.asarray(x, dtype=np.uint16).astype(np.uint32) << 16
        return bits.view(np.float32).astype(np.float64)
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    raise ValueError(dtype)


def ancestors_or_self(parent: Sequence[int]) -> list:
    """anc*(n) for every node of a tree given by its BFS parent array."""
    anc = []
    for n in range(len(parent)):
        path = {n}
        p = int(parent[n])
        while p >= 0:
            path.add(p)
            p = int(parent[p])
        anc.append(path)
    return anc


def verify_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray,
                     ctx_len: Sequence[int], n_q: Sequence[int], num_kv_heads: int,
                     dtype: str = "f32", tree_parent: Optional[Sequence[int]] = None,
                     scale: Optional[float] = None,
                     tree_parents: Optional[Sequence[Sequence[int]]] = None) -> np.ndarray:
    """Verify attention for a packed ragged batch; returns fp64 [Nq, Hq, d].

    q: [Nq, Hq, d]; k, v: [Nkv, Hkv, d]; request i owns query rows
    q0_i .. q0_i + n_i - 1 and KV rows kv0_i .. kv0_i + c_i + n_i - 1, with
    q0 and kv0 the running sums of n_i and c_i + n_i.  tree_parent: one tree
    for every request; tree_parents: request i's tree is tree_parents[i]
    (None for both: chains).
    """
    Q = widen(q, dtype)
    Nq, Hq, d = Q.shape
    Hkv = int(num_kv_heads)
    if Hq % Hkv:
        raise ValueError("query heads must be a multiple of KV heads")
    G = Hq // Hkv
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    out = np.zeros((Nq, Hq, d), dtype=np.float64)
    q0 = kv0 = 0
    for i, (c, n) in enumerate(zip(ctx_len, n_q)):
        c, n = int(c), int(n)
        L = c + n
        par = tree_parents[i] if tree_parents is not None else tree_parent
        if par is None:
            anc = [set(range(j + 1)) for j in range(n)]
        else:
            if len(par) != n:
                raise ValueError("tree size must equal the number of verify nodes")
            anc = ancestors_or_self(par)
        # visibility of each key position to each verify node
        mask = np.zeros((n, L), dtype=bool)
        mask[:, :c] = True
        for j in range(n):
            for t in anc[j]:
                mask[j, c + t] = True
        Kr = widen(k[kv0:kv0 + L], dtype)     # [L, Hkv, d]
        Vr = widen(v[kv0:kv0 + L], dtype)
        for h in range(Hq):
            g = h // G
            s = scale * (Q[q0:q0 + n, h, :] @ Kr[:, g, :].T)     # [n, L]
            s = np.where(mask, s, -np.inf)
            s = s - s.max(axis=1, keepdims=True)
            w = np.exp(s)
            w = w / w.sum(axis=1, keepdims=True)
            out[q0:q0 + n, h, :] = w @ Vr[:, g, :]
        q0 += n
        kv0 += L
    return out


def gather_paged(pool_rows: np.ndarray, block_table: np.ndarray, page_tokens: int, ctx_len, n_q) -> np.ndarray:
    """The packed [Nkv, Hkv, d] rows of a paged cache (the PagedAttention
    layout the paper cites as serving practice, Sec. 6.2): logical KV row t of
    request i is row t % page_tokens of page block_table[i, t // page_tokens]
    of the pool, given here as [num_pages * page_tokens, Hkv, d]."""
    out = []
    for i in range(len(ctx_len)):
        for t in range(int(ctx_len[i]) + int(n_q[i])):
            page = int(block_table[i, t // page_tokens])
            out.append(pool_rows[page * page_tokens + t % page_tokens])
    return np.stack(out)
