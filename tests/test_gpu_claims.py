"""GPU: work items claimed at run time by the bf16 split kernel's later
work-groups, against the same call with every item taken by the work-group
of its own index (bit-identical) and the fp64 oracle.

Work-groups at or above the first round claim the next item from a word in
the workspace that carries the call's tag, so the word is never cleared: a
workspace of random bytes and back-to-back calls on one workspace must give
the same outputs.  Which work-group runs an item changes nothing in its
arithmetic (the split combine sums pieces in piece order), so every setting
is bit-identical to the static launch.  SPEC_ATTN_FIRST_ROUND and
SPEC_ATTN_EXTRA_WG move the first round and the surplus work-groups so that
small batches reach the claims (by default the first round is one
work-group per slot, so only batches of more items than slots claim).
"""
import numpy as np
import pytest
import torch

import parity_util as U
from paper_2505_17074_amd.batch import DeviceBatch, PagedKV, Verifier

pytestmark = pytest.mark.gpu

STATIC = str(1 << 20)     # SPEC_ATTN_FIRST_ROUND above any item count: no claims

CASES = [
    # three-wave items, split and unsplit requests side by side, fused combine
    ("w3_mixed", dict(ctx=[40, 6000, 700, 2100], k=[8, 1, 5, 3], Hq=32, Hkv=8), 512),
    # one-wave items, 20 and 8 pieces per stream
    ("w1_mha", dict(ctx=[5000, 2000, 97], k=[4, 2, 0], Hq=4, Hkv=4), 256),
    # five-wave items, 13-47 pieces: the separate combine kernel, whose
    # request table and row map the split kernel's last work-groups copy
    ("w5_combine_kernel", dict(ctx=[9000, 3000, 12000], k=[8, 8, 8], Hq=64, Hkv=8), 256),
    # a shared token tree, no split
    ("tree", dict(ctx=[0, 50, 300], tree_parent=[-1, 0, 0, 0, 1, 1, 2, 4, 4, 7]), 0),
    # d = 64
    ("d64", dict(ctx=[100, 2500, 33], k=[7, 2, 0], Hq=8, Hkv=2, d=64), 128),
]

# (first round, surplus work-groups): the first item claimed, claims with no
# surplus, a surplus larger than the items, the default surplus
SETTINGS = [("1", "0"), ("1", "40"), ("5", "3"), ("2", None)]


@pytest.fixture
def claims(monkeypatch):
    def set_claims(first, extra):
        monkeypatch.setenv("SPEC_ATTN_FIRST_ROUND", first)
        if extra is None:
            monkeypatch.delenv("SPEC_ATTN_EXTRA_WG", raising=False)
        else:
            monkeypatch.setenv("SPEC_ATTN_EXTRA_WG", extra)
    return set_claims


def _attention(pool, split_kv, junk_seed=None, paged=False, which="attn"):
    b = DeviceBatch(pool, "cuda")
    pk = PagedKV(b, 64, seed=3) if paged else None     # owns the page pools the kernels read
    v = Verifier(b, split_kv=split_kv, attn=pk.attn_args(split_kv) if paged else None)
    if junk_seed is not None:
        g = torch.Generator(device="cuda").manual_seed(junk_seed)
        v._ws.copy_(torch.randint(0, 256, v._ws.shape, dtype=torch.uint8, device="cuda", generator=g))
    v.run(which)
    return v.results()


@pytest.mark.parametrize("name,kw,split", CASES, ids=[c[0] for c in CASES])
def test_claimed_items_match_static_launch(gpu_lib, claims, name, kw, split):
    seed = U.case_seed("claims_" + name)
    pool = U.custom_pool(seed=seed, **kw)
    print(f"[case] claims {name} seed {seed} split_kv {split} static", flush=True)
    claims(STATIC, "0")
    ref = _attention(pool, split)["out"]
    oracle = U.oracle_attention_rows(pool, range(pool.batch))
    r = U.attention_ratios(ref, pool, oracle)
    assert np.isfinite(r).all() and r.max() <= U.ATTN_RTOL, name
    for first, extra in SETTINGS:
        print(f"[case] claims {name} first round {first} surplus {extra}", flush=True)
        claims(first, extra)
        out = _attention(pool, split)["out"]
        assert np.array_equal(out.view(np.uint32), ref.view(np.uint32)), (name, first, extra)
    # a claim word of random bytes starts over at its first claim
    claims("1", "16")
    for junk in (1, 2):
        print(f"[case] claims {name} junk workspace {junk}", flush=True)
        out = _attention(pool, split, junk_seed=junk)["out"]
        assert np.array_equal(out.view(np.uint32), ref.view(np.uint32)), (name, junk)


def test_claims_repeated_calls_and_full_step(gpu_lib, claims):
    """Back-to-back verify steps on one workspace (the claim word keeps the
    previous call's value) give the static launch's outputs every time, the
    acceptance's included."""
    name = "claims_repeat"
    pool = U.custom_pool(ctx=[7000, 150, 16000, 900], k=[8, 3, 8, 5], Hq=32, Hkv=8, seed=U.case_seed(name))
    print(f"[case] {name} static", flush=True)
    claims(STATIC, "0")
    ref = _attention(pool, 384, which="verify")
    claims("3", "24")
    b = DeviceBatch(pool, "cuda")
    v = Verifier(b, split_kv=384)
    for rep in range(4):
        print(f"[case] {name} call {rep}", flush=True)
        b.out.fill_(float("nan"))
        v.run("verify")
        got = v.results()
        assert np.array_equal(got["out"].view(np.uint32), ref["out"].view(np.uint32)), rep
        for key in ("accepted_len", "next_token", "accepted_node"):
            assert np.array_equal(got[key], ref[key]), (rep, key)


def test_claims_paged_cache(gpu_lib, claims):
    """The paged instantiation claims the same way."""
    name = "claims_paged"
    pool = U.custom_pool(ctx=[300, 1200, 40, 5000], k=[5, 7, 3, 7], Hq=8, Hkv=2, seed=U.case_seed(name))
    print(f"[case] {name} static", flush=True)
    claims(STATIC, "0")
    ref = _attention(pool, 256, paged=True)["out"]
    claims("2", "8")
    print(f"[case] {name} claimed", flush=True)
    out = _attention(pool, 256, paged=True)["out"]
    assert np.array_equal(out.view(np.uint32), ref.view(np.uint32))


@pytest.mark.parametrize("paged", [False, True], ids=["packed", "paged"])
def test_claims_at_full_size(gpu_lib, claims, monkeypatch, paged):
    """The 128-request ragged GQA batch at its full size claims by default
    (more items than the device holds work-groups): its outputs equal the
    static launch's bit for bit, and both give every request's sampled rows
    within the oracle's tolerance."""
    from paper_2505_17074_amd import workload as W
    pool = W.make_pool(W.CONFIG_BY_NAME["ragged_gqa_b128"], 0)
    print(f"[case] claims full size ragged_gqa_b128 seed 0 paged {paged} static", flush=True)
    claims(STATIC, "0")
    ref = _attention(pool, 0, paged=paged)["out"]
    print(f"[case] claims full size ragged_gqa_b128 seed 0 paged {paged} default", flush=True)
    monkeypatch.delenv("SPEC_ATTN_FIRST_ROUND", raising=False)
    monkeypatch.delenv("SPEC_ATTN_EXTRA_WG", raising=False)
    out = _attention(pool, 0, paged=paged)["out"]
    assert np.array_equal(out.view(np.uint32), ref.view(np.uint32))
    reqs = [0, 1, pool.batch // 2, pool.batch - 1, int(np.argmax(pool.ctx_len))]
    oracle = U.oracle_attention_rows(pool, reqs)
    r = U.attention_ratios(out, pool, oracle)
    assert np.isfinite(r).all() and r.max() <= U.ATTN_RTOL
