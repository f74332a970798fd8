"""Pins of the fp64 verify-attention oracle against facts outside itself.

Each test checks the oracle against a closed form, an invariant of softmax
attention, or an independent library routine (PyTorch's fp64 scaled
dot-product attention with an explicit boolean mask), chosen so that a
dropped scale, a wrong head map, a wrong mask or a transposed operand fails
at least one of them.
"""
import numpy as np
import pytest
import torch

from oracle import verify_attention, ancestors_or_self

RNG = np.random.default_rng(1234)


def _rand(shape, rng=RNG):
    return rng.standard_normal(shape).astype(np.float32)


def _batch(ctx, n_q, Hq, Hkv, d, rng=RNG):
    Nq = sum(n_q)
    Nkv = sum(c + n for c, n in zip(ctx, n_q))
    return _rand((Nq, Hq, d), rng), _rand((Nkv, Hkv, d), rng), _rand((Nkv, Hkv, d), rng)


def _sdpa(q, k, v, ctx, n_q, Hkv, parent=None, parents=None):
    """Independent reference: torch SDPA in fp64 with repeated KV heads
    (parents: a parent array per request)."""
    Hq = q.shape[1]
    G = Hq // Hkv
    out = np.zeros(q.shape, np.float64)
    q0 = kv0 = 0
    for i, (c, n) in enumerate(zip(ctx, n_q)):
        if parents is not None:
            parent = parents[i]
        L = c + n
        mask = torch.zeros(n, L, dtype=torch.bool)
        mask[:, :c] = True
        if parent is None:
            for j in range(n):
                mask[j, c:c + j + 1] = True
        else:
            for j in range(n):
                node = j
                while node >= 0:
                    mask[j, c + node] = True
                    node = parent[node]
        Q = torch.from_numpy(q[q0:q0 + n].astype(np.float64)).permute(1, 0, 2)        # [Hq, n, d]
        K = torch.from_numpy(k[kv0:kv0 + L].astype(np.float64)).permute(1, 0, 2)
        V = torch.from_numpy(v[kv0:kv0 + L].astype(np.float64)).permute(1, 0, 2)
        K = K.repeat_interleave(G, dim=0)
        V = V.repeat_interleave(G, dim=0)
        O = torch.nn.functional.scaled_dot_product_attention(Q[None], K[None], V[None], attn_mask=mask)
        out[q0:q0 + n] = O[0].permute(1, 0, 2).numpy()
        q0 += n
        kv0 += L
    return out


@pytest.mark.parametrize("Hq,Hkv,d", [(4, 4, 8), (4, 2, 8), (6, 2, 4), (8, 1, 16)])
def test_matches_torch_sdpa_chain(Hq, Hkv, d):
    ctx, n_q = [0, 3, 7, 1], [1, 3, 5, 2]
    q, k, v = _batch(ctx, n_q, Hq, Hkv, d)
    ours = verify_attention(q, k, v, ctx, n_q, Hkv)
    ref = _sdpa(q, k, v, ctx, n_q, Hkv)
    np.testing.assert_allclose(ours, ref, rtol=1e-12, atol=1e-12)


def test_matches_torch_sdpa_tree():
    parent = [-1, 0, 0, 1, 1, 2, 2]
    ctx, n_q = [5, 0, 2], [7, 7, 7]
    q, k, v = _batch(ctx, n_q, 4, 2, 8)
    ours = verify_attention(q, k, v, ctx, n_q, 2, tree_parent=parent)
    ref = _sdpa(q, k, v, ctx, n_q, 2, parent=parent)
    np.testing.assert_allclose(ours, ref, rtol=1e-12, atol=1e-12)


# per-request topologies: a path, a binary tree, a wide root, a lone root,
# a non-binary tree
PER_REQUEST = [[-1, 0, 1, 2], [-1, 0, 0, 1, 1, 2, 2], [-1, 0, 0, 0, 0], [-1], [-1, 0, 0, 1, 1, 1, 3]]


def test_matches_torch_sdpa_per_request_trees():
    ctx = [3, 0, 9, 4, 1]
    n_q = [len(p) for p in PER_REQUEST]
    q, k, v = _batch(ctx, n_q, 4, 2, 8)
    ours = verify_attention(q, k, v, ctx, n_q, 2, tree_parents=PER_REQUEST)
    ref = _sdpa(q, k, v, ctx, n_q, 2, parents=PER_REQUEST)
    np.testing.assert_allclose(ours, ref, rtol=1e-12, atol=1e-12)


def test_per_request_paths_are_chains_and_shared_trees_agree():
    ctx = [3, 0, 9]
    n_q = [4, 2, 5]
    q, k, v = _batch(ctx, n_q, 4, 2, 8)
    paths = [list(range(-1, n - 1)) for n in n_q]
    np.testing.assert_array_equal(verify_attention(q, k, v, ctx, n_q, 2, tree_parents=paths),
                                  verify_attention(q, k, v, ctx, n_q, 2))
    tree = [-1, 0, 0, 1, 2]
    q, k, v = _batch(ctx, [5] * 3, 4, 2, 8)
    np.testing.assert_array_equal(verify_attention(q, k, v, ctx, [5] * 3, 2, tree_parents=[tree] * 3),
                                  verify_attention(q, k, v, ctx, [5] * 3, 2, tree_parent=tree))


def test_single_visible_key_returns_its_value():
    # c = 0 and one verify node: the query sees only its own key, whatever the scores
    q, k, v = _batch([0], [1], 2, 2, 8)
    out = verify_attention(q, k, v, [0], [1], 2)
    np.testing.assert_array_equal(out[0], v[0].astype(np.float64))


def test_two_keys_closed_form_uses_inverse_sqrt_d_scale():
    d = 16
    q, k, v = _batch([1], [1], 1, 1, d)
    out = verify_attention(q, k, v, [1], [1], 1)
    qq, kk, vv = (x.astype(np.float64) for x in (q[0, 0], k[:, 0], v[:, 0]))
    a, b = qq @ kk[0] / 4.0, qq @ kk[1] / 4.0          # 1/sqrt(16)
    expect = (np.exp(a) * vv[0] + np.exp(b) * vv[1]) / (np.exp(a) + np.exp(b))
    np.testing.assert_allclose(out[0, 0], expect, rtol=1e-13)
    out2 = verify_attention(q, k, v, [1], [1], 1, scale=0.5)
    a, b = 0.5 * (qq @ kk[0]), 0.5 * (qq @ kk[1])
    expect2 = (np.exp(a) * vv[0] + np.exp(b) * vv[1]) / (np.exp(a) + np.exp(b))
    np.testing.assert_allclose(out2[0, 0], expect2, rtol=1e-13)


def test_identical_keys_average_visible_values():
    ctx, n_q, Hkv = [4, 2], [3, 4], 1
    q, k, v = _batch(ctx, n_q, 2, Hkv, 8)
    k[:] = k[0]
    out = verify_attention(q, k, v, ctx, n_q, Hkv)
    q0 = kv0 = 0
    for c, n in zip(ctx, n_q):
        for j in range(n):
            vis = list(range(c)) + [c + t for t in range(j + 1)]
            expect = v[kv0 + np.array(vis), 0].astype(np.float64).mean(axis=0)
            for h in range(2):
                np.testing.assert_allclose(out[q0 + j, h], expect, rtol=1e-12, atol=1e-14)
        q0 += n
        kv0 += c + n


def test_constant_values_pass_through():
    ctx, n_q = [3, 9], [2, 5]
    q, k, v = _batch(ctx, n_q, 4, 2, 8)
    z = _rand((2, 8))
    v[:] = z[None]
    out = verify_attention(q, k, v, ctx, n_q, 2)
    for h in range(4):
        np.testing.assert_allclose(out[:, h], np.broadcast_to(z[h // 2].astype(np.float64), out[:, h].shape),
                                   rtol=1e-12)


def test_dominant_score_selects_that_value():
    d = 8
    q, k, v = _batch([6], [1], 1, 1, d)
    q[0, 0] = 0
    q[0, 0, 0] = 1.0
    k[:, 0, 0] = 0.0
    k[3, 0, 0] = 200.0         # exp(200/sqrt(8)) dwarfs the rest
    out = verify_attention(q, k, v, [6], [1], 1)
    np.testing.assert_allclose(out[0, 0], v[3, 0], rtol=1e-12)


def test_invisible_positions_do_not_matter_chain():
    ctx, n_q = [5], [5]
    q, k, v = _batch(ctx, n_q, 2, 1, 8)
    base = verify_attention(q, k, v, ctx, n_q, 1)
    k2, v2 = k.copy(), v.copy()
    k2[5 + 3:] += 10.0
    v2[5 + 3:] -= 7.0           # drafts 3 and 4 are invisible to nodes 0..2
    out = verify_attention(q, k2, v2, ctx, n_q, 1)
    np.testing.assert_array_equal(out[:3], base[:3])
    assert np.abs(out[3:] - base[3:]).max() > 1e-3


def test_invisible_positions_do_not_matter_tree():
    parent = [-1, 0, 0, 1, 1, 2, 2]
    anc = ancestors_or_self(parent)
    assert anc[3] == {0, 1, 3} and anc[6] == {0, 2, 6}
    ctx, n_q = [4], [7]
    q, k, v = _batch(ctx, n_q, 2, 2, 8)
    base = verify_attention(q, k, v, ctx, n_q, 2, tree_parent=parent)
    k2, v2 = k.copy(), v.copy()
    k2[4 + 2] += 5.0            # node 2: visible only to nodes 2, 5, 6
    v2[4 + 2] += 5.0
    out = verify_attention(q, k2, v2, ctx, n_q, 2, tree_parent=parent)
    for j in range(7):
        if j in (2, 5, 6):
            assert np.abs(out[j] - base[j]).max() > 1e-3
        else:
            np.testing.assert_array_equal(out[j], base[j])


def test_gqa_equals_mha_with_repeated_kv():
    ctx, n_q, G = [6, 2], [3, 2], 3
    q, k, v = _batch(ctx, n_q, 6, 2, 8)
    gqa = verify_attention(q, k, v, ctx, n_q, 2)
    mha = verify_attention(q, np.repeat(k, G, axis=1), np.repeat(v, G, axis=1), ctx, n_q, 6)
    np.testing.assert_allclose(gqa, mha, rtol=1e-13, atol=1e-15)
    # the head map is h // G: moving KV head 1 changes only query heads 3..5
    k2 = k.copy()
    k2[:, 1] = _rand(k2[:, 1].shape)
    out = verify_attention(q, k2, v, ctx, n_q, 2)
    np.testing.assert_array_equal(out[:, :3], gqa[:, :3])
    assert np.abs(out[:, 3:] - gqa[:, 3:]).max() > 1e-3


def test_context_order_and_common_key_shift_do_not_matter():
    ctx, n_q = [9], [3]
    q, k, v = _batch(ctx, n_q, 2, 1, 8)
    base = verify_attention(q, k, v, ctx, n_q, 1)
    perm = np.concatenate([RNG.permutation(9), np.arange(9, 12)])
    np.testing.assert_allclose(verify_attention(q, k[perm], v[perm], ctx, n_q, 1), base, rtol=1e-12, atol=1e-14)
    # adding one vector to every key shifts all scores of a query equally (grid values: exact in fp32)
    kg = (np.rint(k * 256) / 256).astype(np.float32)
    shift = (np.rint(_rand((1, 1, 8)) * 256) / 256).astype(np.float32)
    np.testing.assert_allclose(verify_attention(q, kg + shift, v, ctx, n_q, 1),
                               verify_attention(q, kg, v, ctx, n_q, 1), rtol=1e-12, atol=1e-13)


def test_linear_in_values():
    ctx, n_q = [4, 3], [2, 2]
    q, k, v = _batch(ctx, n_q, 2, 1, 8)
    # values on a 2^-8 grid so that v + 2*v2 is exact in fp32 storage
    v = (np.rint(v * 256) / 256).astype(np.float32)
    v2 = (np.rint(_rand(v.shape) * 256) / 256).astype(np.float32)
    a = verify_attention(q, k, v, ctx, n_q, 1)
    b = verify_attention(q, k, v2, ctx, n_q, 1)
    ab = verify_attention(q, k, v + 2 * v2, ctx, n_q, 1)
    np.testing.assert_allclose(ab, a + 2 * b, rtol=1e-12, atol=1e-12)


def test_path_tree_equals_chain():
    ctx, n_q = [3, 5], [4, 4]
    q, k, v = _batch(ctx, n_q, 2, 1, 8)
    chain = verify_attention(q, k, v, ctx, n_q, 1)
    path = verify_attention(q, k, v, ctx, n_q, 1, tree_parent=[-1, 0, 1, 2])
    np.testing.assert_array_equal(chain, path)


def test_bf16_storage_widens_exactly():
    bits = np.array([[[0x3F80, 0xC000, 0x3F81, 0x0000]]], dtype=np.uint16)   # 1, -2, 1.0078125, 0
    out = verify_attention(bits[:, :, :4], bits, bits, [0], [1], 1, dtype="bf16")
    np.testing.assert_array_equal(out[0, 0], [1.0, -2.0, 1.0078125, 0.0])


def _brute(q, k, v, ctx, n_q, Hkv, parent=None):
    """The definition written out with Python loops and math.exp: for request
    i, query head h, node j -- KV head h // G, the visible set (the cached
    positions plus the ancestors-or-self of j, causal for a chain), scores
    scaled by 1/sqrt(d), softmax with the max subtracted, the weighted sum of
    the visible V rows."""
    import math
    Nq, Hq, d = q.shape
    G = Hq // Hkv
    out = np.zeros(q.shape, np.float64)
    q0 = kv0 = 0
    for c, n in zip(ctx, n_q):
        for j in range(n):
            if parent is None:
                anc = set(range(j + 1))
            else:
                anc, a = set(), j
                while a >= 0:
                    anc.add(a)
                    a = parent[a]
            vis = list(range(c)) + [c + t for t in sorted(anc)]
            for h in range(Hq):
                g = h // G
                s = []
                for t in vis:
                    acc = 0.0
                    for e in range(d):
                        acc += float(q[q0 + j, h, e]) * float(k[kv0 + t, g, e])
                    s.append(acc / math.sqrt(d))
                mx = max(s)
                w = [math.exp(x - mx) for x in s]
                tot = sum(w)
                for e in range(d):
                    out[q0 + j, h, e] = sum(wt * float(v[kv0 + t, g, e]) for wt, t in zip(w, vis)) / tot
        q0 += n
        kv0 += c + n
    return out


@pytest.mark.parametrize("Hq,Hkv", [(2, 2), (4, 2)])
def test_matches_brute_force_loops_chain(Hq, Hkv):
    ctx, n_q = [0, 5, 8], [3, 1, 4]
    q, k, v = _batch(ctx, n_q, Hq, Hkv, 8)
    np.testing.assert_allclose(verify_attention(q, k, v, ctx, n_q, Hkv), _brute(q, k, v, ctx, n_q, Hkv),
                               rtol=1e-12, atol=1e-12)


def test_matches_brute_force_loops_tree():
    parent = [-1, 0, 0, 1, 2]
    ctx, n_q = [3, 0], [5, 5]
    q, k, v = _batch(ctx, n_q, 4, 2, 6)
    np.testing.assert_allclose(verify_attention(q, k, v, ctx, n_q, 2, tree_parent=parent),
                               _brute(q, k, v, ctx, n_q, 2, parent=parent), rtol=1e-12, atol=1e-12)


def test_paged_gather_round_trip():
    """Scatter packed rows into pages in a random order, gather them back
    through the block table: the packed rows, exactly (and a page order that
    differs only in its spare pages gathers the same)."""
    from oracle.attention import gather_paged
    rng = np.random.default_rng(3)
    ctx, nq, P = [5, 70, 0, 33], [3, 1, 5, 4], 32
    L = [c + n for c, n in zip(ctx, nq)]
    rows = rng.standard_normal((sum(L), 2, 8))
    pages = [(x + P - 1) // P for x in L]
    num_pages = sum(pages) + 4
    order = rng.permutation(num_pages)
    table = np.zeros((len(L), max(pages)), np.int64)
    pool = np.full((num_pages * P, 2, 8), np.nan)
    k, start = 0, 0
    for i, x in enumerate(L):
        for j in range(pages[i]):
            table[i, j] = order[k]
            k += 1
        for t in range(x):
            pool[table[i, t // P] * P + t % P] = rows[start + t]
        start += x
    np.testing.assert_array_equal(gather_paged(pool, table, P, ctx, nq), rows)
