"""Helpers shared by the GPU parity tests: oracle on request subsets and comparisons.

Tolerances:
  attention   per output row (request, node, head):
              max_e |O_gpu - O_ref| <= 2e-3 * max_e |O_ref|   (bf16 inputs, fp32 accumulation)
  acceptance  accepted length, accepted node and next token bit-exact, except
              requests whose oracle decision path has a uniform within 1e-5 of
              a decision boundary (counted as near ties; their results are only
              checked for validity).
"""
from __future__ import annotations

import dataclasses

import numpy as np

from oracle import verify_accept, verify_attention
from paper_2505_17074_amd import workload as W

ATTN_RTOL = 2e-3


def oracle_attention_rows(pool: W.Pool, reqs) -> dict:
    """fp64 oracle output for the listed requests: {i: [n_i, Hq, d]}."""
    q0, kv0, n_q = pool.q_start, pool.kv_start, pool.n_q
    res = {}
    for i in reqs:
        n, c = int(n_q[i]), int(pool.ctx_len[i])
        res[i] = verify_attention(pool.q[q0[i]:q0[i] + n], pool.k[kv0[i]:kv0[i + 1]], pool.v[kv0[i]:kv0[i + 1]],
                                  [c], [n], pool.num_kv_heads, dtype=pool.qkv_dtype,
                                  tree_parent=pool.tree_parent)
    return res


def attention_ratios(gpu_out: np.ndarray, pool: W.Pool, ref: dict) -> np.ndarray:
    """Row-relative errors max|diff| / max|ref| of every compared row."""
    q0, n_q = pool.q_start, pool.n_q
    out = []
    for i, r in ref.items():
        g = gpu_out[q0[i]:q0[i] + int(n_q[i])].astype(np.float64)
        out.append((np.abs(g - r).max(-1) / np.abs(r).max(-1)).ravel())
    return np.concatenate(out)


def oracle_accept(pool: W.Pool, reqs=None) -> dict:
    return verify_accept(pool.target_logits, pool.draft_probs, pool.draft_tokens, pool.uniforms,
                         pool.n_q, dtype=pool.logit_dtype, tree_parent=pool.tree_parent, requests=reqs)


def compare_accept(gpu: dict, ref: dict, pool: W.Pool, reqs=None):
    """Returns (requests that mismatch outside near ties, number of near ties)."""
    reqs = range(pool.batch) if reqs is None else reqs
    max_len = pool.draft_len if pool.tree_parent is None else np.full(pool.batch, int(pool.draft_len.max()))
    bad, ties = [], 0
    for i in reqs:
        a, t = int(gpu["accepted_len"][i]), int(gpu["next_token"][i])
        if ref["near_tie"][i]:
            ties += 1
            if not (0 <= a <= int(max_len[i]) and 0 <= t < pool.vocab):
                bad.append(i)
            continue
        if (a, t, int(gpu["accepted_node"][i])) != (int(ref["accepted_len"][i]), int(ref["next_token"][i]),
                                                    int(ref["accepted_node"][i])):
            bad.append(i)
    return bad, ties


def custom_pool(ctx, k=None, tree_parent=None, Hq=8, Hkv=2, d=128, V=1000, qkv=W.BF16, logit=W.F32,
                seed=0, sigma=1.0) -> W.Pool:
    """A pool with explicit per-request shapes, drawn with the standard recipe."""
    cfg = W.Config("custom", 99, len(ctx), ("const", 0), ("const", 0), Hq, Hkv, d, qkv, logit, V,
                   ("const", sigma))
    rng = np.random.default_rng(seed)
    ctx = np.asarray(ctx, np.int32)
    B = len(ctx)
    if tree_parent is not None:
        par = np.asarray(tree_parent, np.int32)
        n_q = np.full(B, len(par), np.int64)
        klen = np.full(B, 0, np.int32)
        internal = sorted(set(int(x) for x in par[1:]))
    else:
        par = None
        klen = np.asarray(k, np.int32)
        n_q = klen.astype(np.int64) + 1
    Nq, Nkv = int(n_q.sum()), int((ctx + n_q).sum())
    q = W.storage(rng.standard_normal((Nq, Hq, d), dtype=np.float32), qkv)
    kk = W.storage(rng.standard_normal((Nkv, Hkv, d), dtype=np.float32), qkv)
    vv = W.storage(rng.standard_normal((Nkv, Hkv, d), dtype=np.float32), qkv)
    dl = rng.standard_normal((Nq, V)) * 2.0
    tl = W.storage((dl + sigma * rng.standard_normal((Nq, V))).astype(np.float32), logit)
    q_start = np.concatenate([[0], np.cumsum(n_q)])
    rows, srcs, toks = [], [], []
    for i in range(B):
        n = int(n_q[i])
        loc = list(range(n - 1)) if par is None else internal
        base = len(rows)
        rows.extend(int(q_start[i]) + x for x in loc)
        for node in range(1, n):
            parent = node - 1 if par is None else int(par[node])
            srcs.append(base + loc.index(parent))
    probs64 = np.exp(dl[rows] - dl[rows].max(-1, keepdims=True)) if rows else np.zeros((0, V))
    if rows:
        probs64 /= probs64.sum(-1, keepdims=True)
    probs = W.storage(probs64.astype(np.float32), logit)
    stored = W.as_f32(probs, logit).astype(np.float64)
    for s in srcs:
        cdf = np.cumsum(stored[s]) / stored[s].sum()
        toks.append(min(int(np.searchsorted(cdf, rng.random(), side="right")), V - 1))
    uni = (rng.integers(0, 1 << 24, size=Nq) * 2.0 ** -24).astype(np.float32)
    if par is not None:
        depth = np.zeros(len(par), np.int64)
        for node in range(1, len(par)):
            depth[node] = depth[par[node]] + 1
        klen = np.full(B, int(depth.max()), np.int32)
    return W.Pool(dataclasses.replace(cfg, batch=B), seed, ctx, klen, par, np.full(B, sigma), Hq, Hkv, d, qkv,
                  logit, V, q, kk, vv, tl, probs, np.asarray(toks, np.int32), uni)
