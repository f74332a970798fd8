"""Paged KV cache (block tables) through the C ABI: the split-KV kernel reading
page pools in a random page order must give bit-identical outputs to the
packed layout (the same tiles in the same order), and agree with the oracle
on the rows gathered through the block table."""
import numpy as np
import pytest
import torch

import parity_util as U
from paper_2505_17074_amd import workload as W
from paper_2505_17074_amd.batch import DeviceBatch, PagedKV, Verifier

pytestmark = pytest.mark.gpu


def _check_table(pk, pool):
    """Host-side check before any launch: every entry a request reads is a
    distinct page of the pool."""
    L = pool.ctx_len.astype(np.int64) + pool.n_q.astype(np.int64)
    used = []
    for i in range(pool.batch):
        row = pk.table_np[i, :(L[i] + pk.page_tokens - 1) // pk.page_tokens]
        assert (row >= 0).all() and (row < pk.num_pages).all()
        used.extend(row.tolist())
    assert len(set(used)) == len(used)


def _run(pool, page_tokens, which="verify", split_kv=0, seed=0):
    b = DeviceBatch(pool, "cuda")
    packed = Verifier(b, split_kv=split_kv)
    packed.run(which)
    ref = packed.results()
    pk = PagedKV(b, page_tokens, seed=seed)
    _check_table(pk, pool)
    b.out.fill_(float("nan"))
    paged = Verifier(b, split_kv=split_kv, attn=pk.attn_args(split_kv))
    paged.run(which)
    got = paged.results()
    return ref, got, pk


CASES = [
    ("mha_chain", dict(ctx=[40, 300, 7, 1000], k=[4, 0, 8, 3], Hq=8, Hkv=8)),
    ("gqa_chain", dict(ctx=[300, 1200, 40, 5000], k=[5, 7, 3, 7], Hq=8, Hkv=2)),
    ("gqa_d64", dict(ctx=[100, 2500, 33], k=[7, 2, 0], Hq=8, Hkv=2, d=64)),
    ("tree", dict(ctx=[0, 50, 300], tree_parent=[-1, 0, 0, 0, 1, 1, 2, 4, 4, 7])),
    ("wide_group", dict(ctx=[90, 4000], k=[16, 9], Hq=32, Hkv=2)),
    ("long_single", dict(ctx=[20000], k=[5])),
]


@pytest.mark.parametrize("page_tokens", [32, 64, 96, 160, 256])
@pytest.mark.parametrize("name,kw", CASES, ids=[c[0] for c in CASES])
def test_paged_equals_packed_bitwise(gpu_lib, name, kw, page_tokens):
    seed = U.case_seed(name)
    print(f"[case] paged {name} P={page_tokens} seed {seed}", flush=True)
    pool = U.custom_pool(**kw, seed=seed)
    ref, got, _ = _run(pool, page_tokens)
    assert np.array_equal(got["out"].view(np.uint32), ref["out"].view(np.uint32)), name
    for key in ("accepted_len", "next_token", "accepted_node"):
        assert np.array_equal(got[key], ref[key]), key


@pytest.mark.parametrize("split", [32, 256, 1 << 16])
def test_paged_forced_splits(gpu_lib, split):
    print(f"[case] paged split={split}", flush=True)
    pool = U.custom_pool(ctx=[700, 3000, 64], k=[3, 7, 1], Hq=8, Hkv=2, seed=4)
    ref, got, _ = _run(pool, 64, which="attn", split_kv=split)
    assert np.array_equal(got["out"].view(np.uint32), ref["out"].view(np.uint32))


def test_paged_against_the_oracle(gpu_lib):
    """The oracle on the rows gathered back through the block table from the
    page pools as they sit in device memory."""
    from oracle import verify_attention
    from oracle.attention import gather_paged
    print("[case] paged vs oracle", flush=True)
    pool = U.custom_pool(ctx=[130, 600, 33], k=[4, 6, 2], Hq=8, Hkv=2, seed=8)
    _, got, pk = _run(pool, 64, which="attn", seed=5)
    kp = pk.k.view(torch.int16).cpu().numpy().view(np.uint16)
    vp = pk.v.view(torch.int16).cpu().numpy().view(np.uint16)
    k = gather_paged(kp, pk.table_np, 64, pool.ctx_len, pool.n_q)
    v = gather_paged(vp, pk.table_np, 64, pool.ctx_len, pool.n_q)
    assert np.array_equal(k, pool.k) and np.array_equal(v, pool.v)
    ref = verify_attention(pool.q, k, v, pool.ctx_len, pool.n_q, pool.num_kv_heads, dtype=pool.qkv_dtype)
    r = np.abs(got["out"] - ref).max(-1) / np.abs(ref).max(-1)
    assert r.max() <= U.ATTN_RTOL


@pytest.mark.parametrize("idx,page_tokens", [(1, 32), (3, 64), (4, 128)])
def test_paged_full_size_bitwise(gpu_lib, idx, page_tokens):
    cfg = W.CONFIGS[idx]
    print(f"[case] paged {cfg.name} full size P={page_tokens}, seed 0", flush=True)
    pool = U.full_pool(idx)
    ref, got, _ = _run(pool, page_tokens, which="attn")
    assert np.array_equal(got["out"].view(np.uint32), ref["out"].view(np.uint32)), cfg.name
    torch.cuda.empty_cache()


def test_paged_pool_of_4gib_or_more_equals_packed(gpu_lib):
    """Pools whose byte offsets do not fit 32 bits take the paged build with a
    buffer descriptor per tile; pools that fit take one descriptor per item
    over the pool.  A pool of just over 4 GiB per K and V (the pages the
    batch uses scattered among the spare ones) gives the packed outputs bit
    for bit, as the small pools above do."""
    name = "paged_large_pool"
    seed = U.case_seed(name)
    pool = U.custom_pool(ctx=[300, 1200, 40, 5000], k=[5, 7, 3, 7], Hq=8, Hkv=2, seed=seed)
    b = DeviceBatch(pool, "cuda")
    packed = Verifier(b)
    packed.run("attn")
    ref = packed.results()["out"]
    P = 64
    page_bytes = P * b.k.stride(0) * 2
    spare = (1 << 32) // page_bytes + 8                  # num_pages * page_bytes > 2^32
    print(f"[case] {name} seed {seed} page_tokens {P} spare pages {spare} "
          f"pool {(spare + 200) * page_bytes / 2**30:.2f} GiB per K and V", flush=True)
    pk = PagedKV(b, P, seed=seed, spare=spare)
    assert pk.num_pages * page_bytes > (1 << 32)
    b.out.fill_(float("nan"))
    paged = Verifier(b, attn=pk.attn_args(0))
    paged.run("attn")
    got = paged.results()["out"]
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))
