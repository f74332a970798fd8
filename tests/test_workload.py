"""Seeded synthetic pools: determinism, shapes, ranges and the recipe's structure."""
import numpy as np
import pytest

from paper_2505_17074_amd import workload as W


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -9, -2.5, 0.0, 65504.0], dtype=np.float32)
    b = W.to_bf16_bits(x)
    back = W.bf16_bits_to_f32(b)
    assert back[0] == 1.0
    assert back[1] == 1.0                     # exact tie rounds to even mantissa
    assert back[2] == 1.0 + 2 ** -7           # 1.01171875 rounds up
    assert back[3] == -2.5 and back[4] == 0.0
    r = np.random.default_rng(0).standard_normal(10000).astype(np.float32)
    rb = W.bf16_bits_to_f32(W.to_bf16_bits(r))
    assert np.max(np.abs(rb - r) / np.abs(r)) <= 2 ** -8     # unit roundoff of an 8-bit significand


def test_same_seed_same_bytes():
    a = W.make_pool(W.CONFIGS[0], seed=1)
    b = W.make_pool(W.CONFIGS[0], seed=1)
    c = W.make_pool(W.CONFIGS[0], seed=2)
    for f in ("ctx_len", "draft_len", "q", "k", "v", "target_logits", "draft_probs", "draft_tokens", "uniforms"):
        assert np.array_equal(getattr(a, f), getattr(b, f)), f
    assert not np.array_equal(a.k, c.k)


@pytest.mark.parametrize("idx,batch", [(0, None), (1, 3), (2, 16), (3, 1), (4, 3)])
def test_shapes_and_ranges(idx, batch):
    cfg = W.CONFIGS[idx]
    p = W.make_pool(cfg, seed=0, batch=batch)
    B = p.batch
    n_q = p.n_q
    Nq, Nkv = int(n_q.sum()), int((p.ctx_len + n_q).sum())
    assert p.q.shape == (Nq, cfg.num_q_heads, cfg.head_dim)
    assert p.k.shape == p.v.shape == (Nkv, cfg.num_kv_heads, cfg.head_dim)
    assert p.target_logits.shape == (Nq, cfg.vocab)
    assert p.draft_probs.shape == (int(p.n_internal.sum()), cfg.vocab)
    assert p.draft_tokens.shape == (Nq - B,)
    assert p.uniforms.shape == (Nq,) and p.uniforms.dtype == np.float32
    expect_dtype = np.uint16 if cfg.qkv_dtype == W.BF16 else np.float32
    assert p.k.dtype == expect_dtype
    assert (p.uniforms >= 0).all() and (p.uniforms < 1).all()
    assert np.array_equal(p.uniforms * 2 ** 24, np.floor(p.uniforms * 2 ** 24))
    assert (p.draft_tokens >= 0).all() and (p.draft_tokens < cfg.vocab).all()
    kind = cfg.ctx[0]
    if kind == "uniform":
        assert (p.ctx_len >= cfg.ctx[1]).all() and (p.ctx_len <= cfg.ctx[2]).all()
    if kind == "lognormal":
        assert (p.ctx_len >= cfg.ctx[3]).all() and (p.ctx_len <= cfg.ctx[4]).all()
    if cfg.draft[0] == "uniform":
        assert (p.draft_len >= cfg.draft[1]).all() and (p.draft_len <= cfg.draft[2]).all()
    # every draft token has positive probability under the draft row it was drawn from
    probs = W.as_f32(p.draft_probs, cfg.logit_dtype)
    d0, q0 = p.d_start, p.q_start
    for i in range(B):
        n = int(n_q[i])
        for node in range(1, n):
            par = node - 1 if p.tree_parent is None else int(p.tree_parent[node])
            rank = par if p.tree_parent is None else sorted(set(p.tree_parent[1:].tolist())).index(par)
            tok = int(p.draft_tokens[q0[i] - i + node - 1])
            assert probs[d0[i] + rank, tok] > 0


def test_sigma_mix_and_tree_shape():
    p = W.make_pool(W.CONFIGS[0], seed=0)
    assert list(p.sigma) == [0.5, 1.0, 2.0, 0.5]
    t = W.make_pool(W.CONFIGS[4], seed=0, batch=2)
    assert list(t.tree_parent) == [-1, 0, 0, 1, 1, 2, 2, 3, 3, 4, 4, 5, 5, 6, 6]
    assert t.draft_probs.shape[0] == 2 * 7
    assert (t.ctx_len == 2048).all()


def test_lognormal_context_median():
    cfg = W.CONFIGS[2]
    ctx, klen, sigma = W.request_lengths(cfg, seed=0, batch=4000)
    assert 900 < np.median(ctx) < 1150
    assert ctx.min() >= 32 and ctx.max() <= 8192
    assert 0.3 <= sigma.min() and sigma.max() <= 2.5
    small = W.make_pool(cfg, seed=0, batch=8)
    c8, k8, s8 = W.request_lengths(cfg, seed=0, batch=8)
    assert np.array_equal(small.ctx_len, c8) and np.array_equal(small.draft_len, k8)


def test_accept_bytes_read_model():
    """The acceptance read model: chains read every target row and the draft
    row of each request that rejects; trees read the rows of nodes with
    children, a chosen leaf's row, and a chosen inner node's draft row."""
    from paper_2505_17074_amd import workload as W
    pool = W.make_pool(W.CONFIGS[1], 0, batch=4)
    V, s = pool.vocab, 4
    Nq, B = int(pool.n_q.sum()), pool.batch
    fixed = (Nq - B) * (4 + s) + Nq * 4 + 8 * B
    k = pool.draft_len.astype(np.int64)
    assert W.accept_bytes_read(pool, k) == Nq * V * s + fixed                  # every draft accepted
    assert W.accept_bytes_read(pool, np.zeros(B, np.int64)) == (Nq + B) * V * s + fixed
    assert W.accept_bytes_read(pool, np.zeros(B, np.int64)) == W.workload_bytes(pool)["accept_bytes"]
    tree = W.make_pool(W.CONFIGS[4], 0, batch=3)
    Nq, B, V = int(tree.n_q.sum()), tree.batch, tree.vocab
    fixed = (Nq - B) * (4 + s) + Nq * 4 + 8 * B
    # 15-node binary tree: nodes 0..6 have children; a leaf (14), an inner node (2), the root (0)
    got = W.accept_bytes_read(tree, np.array([14, 2, 0]))
    assert got == (3 * 7 + 1 + 2) * V * s + fixed
