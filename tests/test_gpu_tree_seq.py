"""Sequential sibling verification (SPEC_TREE_SEQUENTIAL) on the GPU against
the oracle: accepted length, accepted node and next token bit-exact except
counted near ties, on the token-tree workload and on irregular trees; and the
exactness identity -- the first emitted token follows the target distribution
-- enumerated through the kernels."""
import itertools

import numpy as np
import pytest

import parity_util as U
from oracle import verify_accept
from paper_2505_17074_amd import binding as B
from paper_2505_17074_amd import workload as W
from paper_2505_17074_amd.batch import DeviceBatch, Verifier

pytestmark = pytest.mark.gpu


def _run_seq(pool):
    b = DeviceBatch(pool, "cuda")
    v = Verifier(b)
    v.acc.tree_rule = B.SPEC_TREE_SEQUENTIAL
    v.run("accept")
    return v.results()


def _check(pool, tag):
    res = _run_seq(pool)
    ref = verify_accept(pool.target_logits, pool.draft_probs, pool.draft_tokens, pool.uniforms, pool.n_q,
                        dtype=pool.logit_dtype, tree_parent=pool.tree_parent, tree_rule="sequential")
    bad, ties = U.compare_accept(res, ref, pool)
    print(f"{tag} B={pool.batch} mean_depth={res['accepted_len'].mean():.3f} near_ties={ties} mismatches={bad}",
          flush=True)
    assert not bad, (tag, bad)
    assert ties <= U.max_near_ties(pool.batch), (tag, ties)
    return res, ref


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_tree_workload_reduced(gpu_lib, seed):
    print(f"[case] sequential tree15 b8 seed {seed}", flush=True)
    _check(W.make_pool(W.CONFIGS[4], seed, batch=8), f"tree15/b8/{seed}")


def test_tree_workload_full_size(gpu_lib):
    print("[case] sequential tree15 full size, seed 0", flush=True)
    res, ref = _check(U.full_pool(4), "tree15/full")
    # the rule reaches the leaves as well as stopping at the root
    assert res["accepted_len"].max() == 3 and res["accepted_len"].min() == 0


@pytest.mark.parametrize("name,kw", [
    ("nonbinary", dict(ctx=[0, 50, 300, 7], tree_parent=[-1, 0, 0, 0, 1, 1, 2, 4, 4, 7])),
    ("wide_root_bf16", dict(ctx=[10, 20, 30], tree_parent=[-1, 0, 0, 0, 0, 0, 1, 2], V=5000, logit=W.BF16)),
    ("vocab_tail", dict(ctx=[5, 6], tree_parent=[-1, 0, 0, 1, 1], V=4100, sigma=2.5)),
], ids=["nonbinary", "wide_root_bf16", "vocab_tail"])
def test_irregular_trees(gpu_lib, name, kw):
    seed = U.case_seed(name)
    print(f"[case] sequential {name} seed {seed}", flush=True)
    _check(U.custom_pool(**kw, seed=seed), name)


def _cells(breaks):
    b = sorted(set([0.0, 1.0] + [float(x) for x in breaks if 0.0 < x < 1.0]))
    return [((lo + hi) / 2.0, hi - lo) for lo, hi in zip(b[:-1], b[1:])]


def test_first_token_distribution_exact_on_gpu(gpu_lib):
    """Two children drafted i.i.d. from q under the root: one request per
    (token pair, uniform cell) combination; weighting each request's first
    emitted token by its probability must give the target distribution."""
    print("[case] sequential vocab-8 enumeration", flush=True)
    V = 8
    rng = np.random.default_rng(23)
    def dist():
        x = rng.random(V) + 0.02
        x = (x / x.sum()).astype(np.float32).astype(np.float64)
        return x / x.sum()
    p0, q0 = dist(), dist()
    q32 = q0.astype(np.float32)
    qd = q32.astype(np.float64)
    runs = [p0]
    for _ in range(2):
        w = np.maximum(0.0, runs[-1] - qd)
        runs.append(w / w.sum())
    fin = np.cumsum(runs[2]) / runs[2].sum()
    cases = []
    for x1, x2 in itertools.product(range(V), repeat=2):
        for (u1, l1), (u2, l2), (uf, lf) in itertools.product(
                _cells([min(1.0, runs[0][x1] / qd[x1])]), _cells([min(1.0, runs[1][x2] / qd[x2])]), _cells(fin)):
            cases.append((x1, x2, u1, u2, uf, qd[x1] * qd[x2] * l1 * l2 * lf))
    n = len(cases)
    pool = U.custom_pool(ctx=[0] * n, tree_parent=[-1, 0, 0], Hq=1, Hkv=1, d=64, V=V)
    child = np.log(np.stack([dist(), dist()])).astype(np.float32)
    pool.target_logits[:] = np.tile(np.concatenate([np.log(p0)[None].astype(np.float32), child]), (n, 1))
    pool.draft_probs[:] = np.tile(q32[None], (n, 1))
    pool.draft_tokens[:] = np.array([[c[0], c[1]] for c in cases]).ravel()
    pool.uniforms[:] = np.array([[c[2], c[3], c[4]] for c in cases], np.float32).ravel()
    out = _run_seq(pool)
    got = np.zeros(V)
    for i, c in enumerate(cases):
        node, length = int(out["accepted_node"][i]), int(out["accepted_len"][i])
        y = (c[0] if node == 1 else c[1]) if length == 1 else int(out["next_token"][i])
        got[y] += c[5]
    np.testing.assert_allclose(got, p0, rtol=0, atol=1e-6)


@pytest.mark.parametrize("groups", [1, 2, 3, 8])
def test_work_groups_per_request(gpu_lib, monkeypatch, groups):
    """The walk split over 1, 2, 3 and 8 work-groups per request (uneven
    slices at 3; 8 slices of one chunk each at the 32000-entry vocabulary),
    every exchange of normalisers and slice totals through the request's
    counter, against the oracle."""
    monkeypatch.setenv("SPEC_SEQ_GROUPS", str(groups))
    print(f"[case] sequential tree15 b16 seed 5, {groups} work-groups per request", flush=True)
    _check(W.make_pool(W.CONFIGS[4], 5, batch=16), f"tree15/b16/groups{groups}")
    seed = U.case_seed("groups_wide_bf16")
    pool = U.custom_pool(ctx=[10, 20, 30, 40], tree_parent=[-1, 0, 0, 0, 0, 0, 1, 2, 2, 2], V=20000, logit=W.BF16,
                         seed=seed, sigma=2.0)
    _check(pool, f"wide/bf16/groups{groups}")


def test_full_step_beside_the_attention(gpu_lib):
    """The sequential rule inside spec_verify: its work-groups run on the side
    stream while the attention's fill the device, so a request's later
    work-groups may start only as attention work-groups finish (the waits are
    bounded well past that).  Three calls on one workspace give the oracle's
    decisions, attention within tolerance, and bit-identical outputs."""
    print("[case] sequential rule in the full verify step, tree15 full size, seed 0", flush=True)
    pool = U.full_pool(4)
    b = DeviceBatch(pool, "cuda")
    v = Verifier(b)
    v.acc.tree_rule = B.SPEC_TREE_SEQUENTIAL
    outs = []
    for _ in range(3):
        b.accepted_len.fill_(-7)
        b.next_token.fill_(-7)
        v.run("verify")
        outs.append(v.results())
    ref = verify_accept(pool.target_logits, pool.draft_probs, pool.draft_tokens, pool.uniforms, pool.n_q,
                        dtype=pool.logit_dtype, tree_parent=pool.tree_parent, tree_rule="sequential")
    bad, ties = U.compare_accept(outs[0], ref, pool)
    print(f"step/sequential B={pool.batch} near_ties={ties} mismatches={bad}", flush=True)
    assert not bad and ties <= U.max_near_ties(pool.batch)
    for o in outs[1:]:
        for key in ("accepted_len", "next_token", "accepted_node"):
            assert np.array_equal(o[key], outs[0][key]), key
        assert np.array_equal(o["out"].view(np.uint32), outs[0]["out"].view(np.uint32))
    sample = [0, pool.batch // 2, pool.batch - 1]
    r = U.attention_ratios(outs[0]["out"], pool, U.oracle_attention_rows(pool, sample))
    assert np.isfinite(r).all() and r.max() <= U.ATTN_RTOL
