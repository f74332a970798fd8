"""Per-request token trees (each request its own topology, the SpecInfer
setup of one speculated tree per request, Sec. 5.1) on the GPU against the
fp64 oracle, through the C ABI: attention within the row-relative tolerance,
accepted length, node and next token bit-exact except counted near ties,
under both tree rules; the same inputs in the shared-tree and chain forms
give bit-identical outputs."""
import copy

import numpy as np
import pytest
import torch

import parity_util as U
from paper_2505_17074_amd import binding as B
from paper_2505_17074_amd import workload as W
from paper_2505_17074_amd.batch import DeviceBatch, PagedKV, Verifier

pytestmark = pytest.mark.gpu

# a path, a binary tree, a wide root, a lone root, a non-binary tree, the
# 15-node binary tree, a 32-node chain-like tree
MIXED = [[-1, 0, 1, 2], [-1, 0, 0, 1, 1, 2, 2], [-1, 0, 0, 0, 0, 0], [-1], [-1, 0, 0, 1, 1, 1, 3],
         W.full_binary_tree_parents(2, 4).tolist(), [-1] + [max(0, n - 2) for n in range(1, 32)]]


def _random_trees(rng, B, max_nodes=32):
    out = []
    for _ in range(B):
        n = int(rng.integers(1, max_nodes + 1))
        out.append([-1] + [int(rng.integers(0, m)) for m in range(1, n)])
    return out


def _run(pool, which="verify", rule=B.SPEC_TREE_INDEPENDENT):
    b = DeviceBatch(pool, "cuda")
    v = Verifier(b)
    v.acc.tree_rule = rule
    v.run(which)
    return v.results()


def _check(pool, res, tag, rule="independent", attention=True):
    if attention:
        ref = U.oracle_attention_rows(pool, range(pool.batch))
        r = U.attention_ratios(res["out"], pool, ref)
        print(f"{tag} attention rows={r.size} worst={r.max():.3e}", flush=True)
        assert np.isfinite(r).all() and r.max() <= U.ATTN_RTOL, tag
    ref = U.oracle_accept(pool, tree_rule=rule)
    bad, ties = U.compare_accept(res, ref, pool)
    print(f"{tag} accept ({rule}) B={pool.batch} mean_depth={res['accepted_len'].mean():.3f} "
          f"near_ties={ties} mismatches={bad}", flush=True)
    assert not bad, (tag, bad)
    assert ties <= U.max_near_ties(pool.batch), (tag, ties)


@pytest.mark.parametrize("logit", [W.F32, W.BF16])
def test_mixed_topologies_against_the_oracle(gpu_lib, logit):
    seed = U.case_seed(f"mixed_trees_{logit}")
    print(f"[case] per-request trees, mixed topologies, logits {logit}, seed {seed}", flush=True)
    pool = U.custom_pool(ctx=[0, 37, 300, 5, 1200, 64, 2000], tree_parents=MIXED, Hq=8, Hkv=2, V=3000,
                         logit=logit, seed=seed)
    res = _run(pool)
    _check(pool, res, "mixed/indep")
    _check(pool, _run(pool, "accept", B.SPEC_TREE_SEQUENTIAL), "mixed/seq", rule="sequential", attention=False)


@pytest.mark.parametrize("seed", [0, 1])
def test_random_trees_tree_workload_shape(gpu_lib, seed):
    """The token-tree workload's shape (GQA 32/8 heads, 2048-token contexts,
    vocabulary 32000) with a random tree of 1-32 nodes per request."""
    print(f"[case] per-request random trees, 16 requests, seed {seed}", flush=True)
    rng = np.random.default_rng(seed)
    trees = _random_trees(rng, 16)
    pool = U.custom_pool(ctx=[2048] * 16, tree_parents=trees, Hq=32, Hkv=8, V=32000, seed=seed, sigma=0.7)
    _check(pool, _run(pool), f"random/{seed}")
    _check(pool, _run(pool, "accept", B.SPEC_TREE_SEQUENTIAL), f"random/{seed}/seq", rule="sequential",
           attention=False)


def test_same_tree_per_request_equals_shared_tree(gpu_lib):
    print("[case] per-request copies of one tree == the shared tree", flush=True)
    tree = W.full_binary_tree_parents(2, 4)
    shared = U.custom_pool(ctx=[100, 0, 2500, 31], tree_parent=tree, Hq=8, Hkv=2, V=5000, seed=5)
    per = copy.copy(shared)
    per.tree_parent = None
    per.tree_parents = [tree.tolist()] * shared.batch
    for rule in (B.SPEC_TREE_INDEPENDENT, B.SPEC_TREE_SEQUENTIAL):
        a, b = _run(shared, rule=rule), _run(per, rule=rule)
        for key in a:
            assert np.array_equal(np.asarray(a[key]).view(np.uint8), np.asarray(b[key]).view(np.uint8)), (rule, key)


def test_paths_per_request_equal_chains(gpu_lib):
    print("[case] per-request paths == chains", flush=True)
    chain = U.custom_pool(ctx=[3, 40, 700, 1, 0], k=[4, 0, 8, 2, 16], Hq=8, Hkv=2, V=4100, seed=9, sigma=0.3)
    per = copy.copy(chain)
    per.tree_parents = [list(range(-1, int(k))) for k in chain.draft_len]
    a, b = _run(chain), _run(per)
    for key in a:
        assert np.array_equal(np.asarray(a[key]).view(np.uint8), np.asarray(b[key]).view(np.uint8)), key


@pytest.mark.parametrize("rule", ["independent", "sequential"])
def test_hand_packed_trees(gpu_lib, rule):
    print(f"[case] per-request trees by hand, {rule}", flush=True)
    inp, expect = U.hand_packed_trees()
    pool = U.custom_pool(ctx=inp["ctx"], tree_parents=inp["parents"], Hq=1, Hkv=1, d=64, V=4)
    for key in ("target_logits", "draft_probs", "draft_tokens", "uniforms"):
        getattr(pool, key)[:] = inp[key]
    res = _run(pool, "accept", B.SPEC_TREE_SEQUENTIAL if rule == "sequential" else B.SPEC_TREE_INDEPENDENT)
    for key, val in expect[rule].items():
        assert res[key].tolist() == val, (rule, key, res[key])


def test_paged_per_request_trees_equal_packed(gpu_lib):
    print("[case] per-request trees over a paged KV cache == packed", flush=True)
    pool = U.custom_pool(ctx=[0, 37, 300, 5, 1200, 64, 2000], tree_parents=MIXED, Hq=8, Hkv=2, V=1000, seed=3)
    ref = _run(pool, "attn")
    b = DeviceBatch(pool, "cuda")
    pk = PagedKV(b, 64, seed=2)                 # owns the page pools the kernels read
    v = Verifier(b, attn=pk.attn_args())
    v.run("attn")
    got = v.results()
    assert np.array_equal(got["out"].view(np.uint32), ref["out"].view(np.uint32))
    del v, pk, b
