"""Seeded synthetic verify-step workloads (input generation only).

This module draws the inputs of one batched speculative-decoding verify step:
per-request context lengths and draft lengths, the query/key/value tensors of
the target model's attention layer, the draft model's token distributions and
sampled draft tokens, the target model's logits, and the uniforms that drive
acceptance and the final sample.  It holds none of the verify step's own
arithmetic (no attention, no target softmax, no acceptance test, no residual
sample): both the HIP path and the CPU oracle consume the arrays it returns.

The draft model's outputs are inputs of the verify step, so generating them
(a softmax of draft logits, a categorical draw of each draft token) belongs
here; the paper's speculative-decoding background (Sec. 2.2) fixes what they
are: the SSM proposes tokens sampled from its own distribution, and the LLM
scores every proposed position in one forward pass.

Workload shapes stand in for the paper's evaluation (Sec. 5.1: LLaMA-68M
drafting for LLaMA-7B on three public prompt datasets, which are not used
here).  Random draws come from ``numpy.random.Generator(PCG64)`` seeded by
``SeedSequence([config_index, seed])`` in a fixed order:
context lengths, draft lengths, noise scales, Q, K, V, draft logits, target
noise, draft tokens, verify uniforms.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np

F32 = "f32"
BF16 = "bf16"


# --------------------------------------------------------------------------
# storage-format helpers (bf16 is stored as its raw uint16 bit pattern)
# --------------------------------------------------------------------------
def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round-to-nearest-even), return bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    nan = (u & 0x7FFFFFFF) > 0x7F800000
    rounded = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    if nan.any():
        rounded[nan] = 0x7FC0
    return rounded


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def storage(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == F32:
        return np.ascontiguousarray(x, dtype=np.float32)
    if dtype == BF16:
        return to_bf16_bits(x)
    raise ValueError(dtype)


def as_f32(x: np.ndarray, dtype: str) -> np.ndarray:
    """Stored values widened to float32 (exact for both storage formats)."""
    return bf16_bits_to_f32(x) if dtype == BF16 else np.asarray(x, np.float32)


# --------------------------------------------------------------------------
# configurations
# --------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    index: int
    batch: int
    ctx: tuple            # ("uniform", lo, hi) | ("lognormal", median, sigma, lo, hi) | ("const", c)
    draft: tuple          # ("const", k) | ("uniform", lo, hi) | ("tree", branching, depth)
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    qkv_dtype: str
    logit_dtype: str
    vocab: int
    sigma: tuple          # ("cyclic", values...) | ("uniform", lo, hi) | ("const", s)
    draft_logit_std: float = 2.0

    @property
    def is_tree(self) -> bool:
        return self.draft[0] == "tree"


CONFIGS = [
    # tiny fp32 verify step: parity-sized, finishes on the CPU oracle in seconds
    Config("tiny_f32", 0, 4, ("uniform", 64, 256), ("const", 4), 8, 8, 64,
           F32, F32, 1024, ("cyclic", 0.5, 1.0, 2.0)),
    # LLaMA-7B-shaped MHA verify (the paper's target model, Sec. 5.1)
    Config("mha7b_b32", 1, 32, ("uniform", 512, 2048), ("const", 4), 32, 32, 128,
           BF16, F32, 32000, ("cyclic", 0.5, 1.0, 2.0)),
    # many-request ragged GQA batch with per-request (adaptive) draft length
    Config("ragged_gqa_b128", 2, 128, ("lognormal", 1024, 1.0, 32, 8192), ("uniform", 1, 8),
           32, 8, 128, BF16, F32, 32000, ("uniform", 0.3, 2.5)),
    # long-context GQA verify with a 128256-entry vocabulary in bf16
    Config("long_gqa_b8", 3, 8, ("uniform", 16384, 32768), ("const", 8), 64, 8, 128,
           BF16, BF16, 128256, ("const", 1.0)),
    # token-tree verification: binary tree of depth 4 (15 nodes, root = last accepted token)
    Config("tree15_b64", 4, 64, ("const", 2048), ("tree", 2, 4), 32, 8, 128,
           BF16, F32, 32000, ("cyclic", 0.5, 1.0, 2.0)),
]
CONFIG_BY_NAME = {c.name: c for c in CONFIGS}


def full_binary_tree_parents(branching: int, depth: int) -> np.ndarray:
    """BFS parent array of a complete tree; node 0 is the root (parent -1)."""
    n = sum(branching ** d for d in range(depth))
    par = np.full(n, -1, dtype=np.int32)
    for node in range(1, n):
        par[node] = (node - 1) // branching
    return par


def chain_parents(n: int) -> np.ndarray:
    par = np.arange(-1, n - 1, dtype=np.int32)
    return par


# --------------------------------------------------------------------------
# the pool
# --------------------------------------------------------------------------
@dataclasses.dataclass
class Pool:
    cfg: Optional[Config]
    seed: int
    ctx_len: np.ndarray          # int32 [B]
    draft_len: np.ndarray        # int32 [B] (chain k_i; for a tree: depth of the deepest node)
    tree_parent: Optional[np.ndarray]   # int32 [n_nodes] shared by the batch, or None (chain)
    sigma: np.ndarray            # float64 [B] (metadata: target-noise scale)
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    qkv_dtype: str
    logit_dtype: str
    vocab: int
    q: np.ndarray                # [Nq, Hq, d] f32 or bf16 bits
    k: np.ndarray                # [Nkv, Hkv, d]
    v: np.ndarray                # [Nkv, Hkv, d]
    target_logits: np.ndarray    # [Nq, V]
    draft_probs: np.ndarray      # [Nd, V]
    draft_tokens: np.ndarray     # int32 [Nq - B]
    uniforms: np.ndarray         # float32 [Nq]
    tree_parents: Optional[list] = None   # per request, its own BFS parent array (instead of tree_parent)
    hidden: Optional[np.ndarray] = None   # LM-head inputs (make_lm_head_pool): [Nq, K] bf16 bits
    weight: Optional[np.ndarray] = None   # [V, K] bf16 bits

    @property
    def batch(self) -> int:
        return int(self.ctx_len.shape[0])

    @property
    def is_tree(self) -> bool:
        return self.tree_parent is not None or self.tree_parents is not None

    def parents_of(self, i: int):
        """Request i's tree (BFS parent array), or None for a chain."""
        return self.tree_parents[i] if self.tree_parents is not None else self.tree_parent

    @property
    def n_q(self) -> np.ndarray:
        if self.tree_parents is not None:
            return np.array([len(p) for p in self.tree_parents], dtype=np.int64)
        if self.tree_parent is not None:
            return np.full(self.batch, len(self.tree_parent), dtype=np.int64)
        return self.draft_len.astype(np.int64) + 1

    @property
    def n_internal(self) -> np.ndarray:
        """Draft-probability rows per request (nodes that have children)."""
        if self.tree_parents is not None:
            return np.array([len(set(int(x) for x in p[1:])) for p in self.tree_parents], dtype=np.int64)
        if self.tree_parent is not None:
            ni = len(set(int(p) for p in self.tree_parent[1:]))
            return np.full(self.batch, ni, dtype=np.int64)
        return self.draft_len.astype(np.int64)

    @property
    def q_start(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.n_q)]).astype(np.int64)

    @property
    def kv_start(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.ctx_len.astype(np.int64) + self.n_q)]).astype(np.int64)

    @property
    def d_start(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.n_internal)]).astype(np.int64)


def _draw_ctx(rng, cfg: Config) -> np.ndarray:
    kind = cfg.ctx[0]
    if kind == "uniform":
        return rng.integers(cfg.ctx[1], cfg.ctx[2] + 1, size=cfg.batch).astype(np.int32)
    if kind == "lognormal":
        _, median, s, lo, hi = cfg.ctx
        c = np.rint(rng.lognormal(mean=math.log(median), sigma=s, size=cfg.batch))
        return np.clip(c, lo, hi).astype(np.int32)
    if kind == "const":
        return np.full(cfg.batch, cfg.ctx[1], dtype=np.int32)
    raise ValueError(kind)


def _draw_draft_len(rng, cfg: Config) -> np.ndarray:
    kind = cfg.draft[0]
    if kind == "const":
        return np.full(cfg.batch, cfg.draft[1], dtype=np.int32)
    if kind == "uniform":
        return rng.integers(cfg.draft[1], cfg.draft[2] + 1, size=cfg.batch).astype(np.int32)
    if kind == "tree":
        return np.full(cfg.batch, cfg.draft[2] - 1, dtype=np.int32)
    raise ValueError(kind)


def _draw_sigma(rng, cfg: Config) -> np.ndarray:
    kind = cfg.sigma[0]
    if kind == "cyclic":
        vals = np.array(cfg.sigma[1:], dtype=np.float64)
        return vals[np.arange(cfg.batch) % len(vals)]
    if kind == "uniform":
        return rng.uniform(cfg.sigma[1], cfg.sigma[2], size=cfg.batch)
    if kind == "const":
        return np.full(cfg.batch, float(cfg.sigma[1]))
    raise ValueError(kind)


def _normal(rng, shape, dtype: str, scale: float = 1.0) -> np.ndarray:
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if scale != 1.0:
        x *= np.float32(scale)
    return storage(x, dtype)


def _softmax_rows(x: np.ndarray) -> np.ndarray:
    x = x - x.max(axis=-1, keepdims=True)
    e = np.exp(x)
    return e / e.sum(axis=-1, keepdims=True)


def _categorical(rng, probs: np.ndarray) -> np.ndarray:
    """One draw per row from the (stored) draft distribution of that row."""
    p = np.asarray(probs, dtype=np.float64)
    cdf = np.cumsum(p, axis=-1)
    cdf /= cdf[:, -1:]
    u = rng.random(p.shape[0])
    tok = np.array([np.searchsorted(cdf[r], u[r], side="right") for r in range(p.shape[0])])
    tok = np.minimum(tok, p.shape[1] - 1)
    # never emit a token the draft model gives zero probability
    for r in range(p.shape[0]):
        while p[r, tok[r]] <= 0.0:
            tok[r] -= 1
    return tok.astype(np.int32)


def _rng(cfg: Config, seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([cfg.index, seed])))


def _draw_request_scalars(rng, cfg: Config):
    ctx = _draw_ctx(rng, cfg)
    klen = _draw_draft_len(rng, cfg)
    sigma = _draw_sigma(rng, cfg)
    return ctx, klen, sigma


def request_lengths(cfg: Config, seed: int = 0, batch: Optional[int] = None):
    """The per-request (context length, draft length, noise scale) draws alone.

    Identical to the first draws of ``make_pool`` with the same arguments,
    without materialising any tensor.
    """
    if batch is not None:
        cfg = dataclasses.replace(cfg, batch=int(batch))
    return _draw_request_scalars(_rng(cfg, seed), cfg)


def make_pool(cfg: Config, seed: int = 0, batch: Optional[int] = None) -> Pool:
    """Draw the seeded synthetic verify-step inputs of one configuration.

    ``batch`` (optional) overrides the number of requests: the result is a
    separate, smaller workload drawn with the same recipe, not a slice of the
    full-size one.
    """
    if batch is not None:
        cfg = dataclasses.replace(cfg, batch=int(batch))
    rng = _rng(cfg, seed)
    B = cfg.batch
    ctx, klen, sigma = _draw_request_scalars(rng, cfg)

    parent = None
    if cfg.is_tree:
        parent = full_binary_tree_parents(cfg.draft[1], cfg.draft[2])
        n_q = np.full(B, len(parent), dtype=np.int64)
    else:
        n_q = klen.astype(np.int64) + 1
    Nq = int(n_q.sum())
    Nkv = int((ctx.astype(np.int64) + n_q).sum())
    Hq, Hkv, d, V = cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim, cfg.vocab

    q = _normal(rng, (Nq, Hq, d), cfg.qkv_dtype)
    k = _normal(rng, (Nkv, Hkv, d), cfg.qkv_dtype)
    v = _normal(rng, (Nkv, Hkv, d), cfg.qkv_dtype)

    # one draft-logit row per verify node (the last one feeds only the target row)
    draft_logits = rng.standard_normal(size=(Nq, V)) * cfg.draft_logit_std
    noise = rng.standard_normal(size=(Nq, V))
    q_start = np.concatenate([[0], np.cumsum(n_q)])
    sig_rows = np.repeat(sigma, n_q)
    target = draft_logits + noise * sig_rows[:, None]
    target_logits = storage(target.astype(np.float32), cfg.logit_dtype)

    # draft distributions: rows of nodes that have children, stored in the logit dtype
    if parent is None:
        internal_local = [np.arange(int(kk)) for kk in klen]
    else:
        internal = sorted(set(int(p) for p in parent[1:]))
        internal_local = [np.array(internal)] * B
    rows = np.concatenate([q_start[i] + internal_local[i] for i in range(B)]).astype(np.int64) \
        if B else np.zeros(0, np.int64)
    probs64 = _softmax_rows(draft_logits[rows]) if rows.size else np.zeros((0, V))
    draft_probs = storage(probs64.astype(np.float32), cfg.logit_dtype)
    del draft_logits, noise, target

    # draft tokens: node n (n >= 1) is drawn from its parent's stored draft row
    stored_probs = as_f32(draft_probs, cfg.logit_dtype).astype(np.float64)
    d_start = np.concatenate([[0], np.cumsum([len(x) for x in internal_local])])
    src_rows = []
    for i in range(B):
        nodes = int(n_q[i])
        if parent is None:
            par_local = np.arange(nodes - 1)                     # node j+1's parent is j
        else:
            par_local = parent[1:]
        rank = {int(n): r for r, n in enumerate(internal_local[i])}
        src_rows.extend(int(d_start[i]) + rank[int(p)] for p in par_local)
    src_rows = np.asarray(src_rows, dtype=np.int64)
    draft_tokens = _categorical(rng, stored_probs[src_rows]) if src_rows.size else np.zeros(0, np.int32)

    uniforms = (rng.integers(0, 1 << 24, size=Nq).astype(np.float64) * 2.0 ** -24).astype(np.float32)

    return Pool(cfg, seed, ctx, klen, parent, sigma, Hq, Hkv, d, cfg.qkv_dtype, cfg.logit_dtype, V,
                q, k, v, target_logits, draft_probs, draft_tokens, uniforms)


def workload_bytes(pool: Pool) -> dict:
    """Algorithmic bytes and flops of one verify step over this pool.

    Attention: K and V rows once, Q once, the fp32 output once.  Acceptance:
    every target-logit row once, plus one draft-probability row per request
    (the row at the first rejection; an upper bound that assumes every request
    rejects), the draft ids, the uniforms and the outputs.
    """
    s_kv = 4 if pool.qkv_dtype == F32 else 2
    s_l = 4 if pool.logit_dtype == F32 else 2
    n_q = pool.n_q
    Nq = int(n_q.sum())
    Nkv = int((pool.ctx_len.astype(np.int64) + n_q).sum())
    d, Hq, Hkv, V, B = pool.head_dim, pool.num_q_heads, pool.num_kv_heads, pool.vocab, pool.batch
    attn_bytes = Nkv * Hkv * d * 2 * s_kv + Nq * Hq * d * s_kv + Nq * Hq * d * 4
    flops = 0
    for i in range(B):
        c, n, par = int(pool.ctx_len[i]), int(n_q[i]), pool.parents_of(i)
        if par is None:
            vis = n * (n + 1) // 2
        else:
            depth = np.zeros(len(par), np.int64)
            for m in range(1, len(par)):
                depth[m] = depth[par[m]] + 1
            vis = int(sum(depth[j] + 1 for j in range(len(par))))
        flops += 4 * d * Hq * (c * n + vis)
    acc_bytes = Nq * V * s_l + B * V * s_l + (Nq - B) * (4 + s_l) + Nq * 4 + 8 * B
    return {"attn_bytes": int(attn_bytes), "attn_flops": int(flops), "accept_bytes": int(acc_bytes),
            "Nq": Nq, "Nkv": Nkv}


def accept_bytes_read(pool: Pool, accepted_node: np.ndarray) -> int:
    """Bytes the acceptance kernels read for this step's outcome (independent
    rule).  Chains: every target row once.  Trees: the rows of nodes with
    children once (their normalisers enter the tests), and the chosen node's
    row where it is a leaf.  Plus the draft row of each chosen node that has
    children (the residual), the draft ids and their draft probabilities,
    the uniforms and the outputs."""
    s_l = 4 if pool.logit_dtype == F32 else 2
    n_q = pool.n_q
    Nq, V, B = int(n_q.sum()), pool.vocab, pool.batch
    node = np.asarray(accepted_node, np.int64)
    if pool.tree_parents is not None:
        # per-request trees: every row's statistics are taken
        rows, qrows = Nq, 0
        for i in range(B):
            par = np.asarray(pool.tree_parents[i])
            inner = np.zeros(len(par), bool)
            inner[par[1:]] = True
            qrows += int(inner[node[i]])
    elif pool.tree_parent is not None:
        par = pool.tree_parent
        inner = np.zeros(len(par), bool)
        inner[par[1:]] = True
        rows = B * int(inner.sum()) + int((~inner[node]).sum())
        qrows = int(inner[node].sum())
    else:
        rows = Nq
        qrows = int((node < pool.draft_len).sum())
    return int((rows + qrows) * V * s_l + (Nq - B) * (4 + s_l) + Nq * 4 + 8 * B)


# hidden size of the target model behind each workload (LLaMA-7B-like 4096;
# the 64-head long-context model 8192)
LM_HIDDEN = {"tiny_f32": 256, "mha7b_b32": 4096, "ragged_gqa_b128": 4096, "long_gqa_b8": 8192, "tree15_b64": 4096}


def make_lm_head_pool(cfg: Config, seed: int = 0, batch: Optional[int] = None,
                      hidden_dim: Optional[int] = None, vocab: Optional[int] = None) -> Pool:
    """A workload's acceptance inputs with the target logits left to the LM
    head: the verify positions' final hidden states [Nq, K] ~ N(0, 1) and the
    LM head's weights [V, K] ~ N(0, 4 / K), both stored in bf16, so that the
    logits have a standard deviation of about 2 (the draft-logit scale of
    make_pool).  The draft model is emulated as an LM head of its own over
    the same hidden states, weights W + N(0, 1 / K) (the target's plus noise),
    plus N(0, sigma_i^2) on its logits with the workload's per-request sigma;
    its distributions are stored in the logit dtype and the draft tokens
    drawn from them.  Q, K and V are not drawn (empty); target_logits is a
    zero buffer of the right shape for the LM head to fill.  Draw order:
    request scalars, hidden states, weights, draft-weight noise (by blocks of
    8192 vocabulary rows), draft-logit noise, draft tokens, uniforms."""
    if batch is not None:
        cfg = dataclasses.replace(cfg, batch=int(batch))
    if vocab is not None:
        cfg = dataclasses.replace(cfg, vocab=int(vocab))
    K = int(hidden_dim or LM_HIDDEN.get(cfg.name, 4096))
    rng = _rng(cfg, seed)
    B, V = cfg.batch, cfg.vocab
    ctx, klen, sigma = _draw_request_scalars(rng, cfg)
    parent = full_binary_tree_parents(cfg.draft[1], cfg.draft[2]) if cfg.is_tree else None
    n_q = np.full(B, len(parent), np.int64) if parent is not None else klen.astype(np.int64) + 1
    Nq = int(n_q.sum())
    hidden = storage(rng.standard_normal((Nq, K), dtype=np.float32), BF16)
    weight = storage(rng.standard_normal((V, K), dtype=np.float32) * np.float32(2.0 / math.sqrt(K)), BF16)
    q_start = np.concatenate([[0], np.cumsum(n_q)])
    if parent is None:
        internal_local = [np.arange(int(kk)) for kk in klen]
    else:
        internal = sorted(set(int(p) for p in parent[1:]))
        internal_local = [np.array(internal)] * B
    rows = np.concatenate([q_start[i] + internal_local[i] for i in range(B)]).astype(np.int64) \
        if B else np.zeros(0, np.int64)
    Hr = bf16_bits_to_f32(hidden[rows]) if rows.size else np.zeros((0, K), np.float32)
    z = np.zeros((rows.size, V), np.float32)
    for v0 in range(0, V, 8192):
        wb = bf16_bits_to_f32(weight[v0:v0 + 8192])
        wb = wb + rng.standard_normal(wb.shape, dtype=np.float32) * np.float32(1.0 / math.sqrt(K))
        z[:, v0:v0 + 8192] = Hr @ wb.T
    req_of_row = np.repeat(np.arange(B), [len(x) for x in internal_local])
    z = z.astype(np.float64) + rng.standard_normal(z.shape) * sigma[req_of_row][:, None]
    draft_probs = storage(_softmax_rows(z).astype(np.float32), cfg.logit_dtype) if rows.size \
        else np.zeros((0, V), np.uint16 if cfg.logit_dtype == BF16 else np.float32)
    stored = as_f32(draft_probs, cfg.logit_dtype).astype(np.float64)
    d_start = np.concatenate([[0], np.cumsum([len(x) for x in internal_local])])
    src_rows = []
    for i in range(B):
        par_local = np.arange(int(n_q[i]) - 1) if parent is None else parent[1:]
        rank = {int(n): r for r, n in enumerate(internal_local[i])}
        src_rows.extend(int(d_start[i]) + rank[int(p)] for p in par_local)
    src_rows = np.asarray(src_rows, dtype=np.int64)
    draft_tokens = _categorical(rng, stored[src_rows]) if src_rows.size else np.zeros(0, np.int32)
    uniforms = (rng.integers(0, 1 << 24, size=Nq).astype(np.float64) * 2.0 ** -24).astype(np.float32)
    empty = np.zeros((0, cfg.num_q_heads, cfg.head_dim), np.float32)
    empty_kv = np.zeros((0, cfg.num_kv_heads, cfg.head_dim), np.float32)
    target = np.zeros((Nq, V), np.uint16 if cfg.logit_dtype == BF16 else np.float32)
    return Pool(cfg, seed, ctx, klen, parent, sigma, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim,
                cfg.qkv_dtype, cfg.logit_dtype, V, empty, empty_kv, empty_kv, target, draft_probs,
                draft_tokens, uniforms, hidden=hidden, weight=weight)
