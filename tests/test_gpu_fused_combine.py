"""GPU: the split combine done inside the bf16 split kernel by each split
stream's last piece, against the fp64 oracle.

The pieces of a (request, KV head, head group) stream check in on a counter
that carries the call's tag, so the counters are never cleared: a workspace
full of junk must give the same outputs as a clean one.  Where a stream's
combine data (rows x pieces (m, l) pairs) does not fit the kernel's LDS, or
its partial block is above the planner's limit, the separate combine kernel
runs instead; those paths are checked too.
"""
import numpy as np
import pytest
import torch

import parity_util as U
from paper_2505_17074_amd.batch import DeviceBatch, Verifier

pytestmark = pytest.mark.gpu

ANY = str(1 << 40)      # SPEC_FUSED_COMBINE_MAX_BYTES: fuse every stream that fits the LDS
CASES = [
    # five-wave items (8 heads x 9 positions = 72 rows), 13-47 pieces per
    # stream: 0.5-1.7 MB per stream, fused only when the limit is lifted
    ("w5_many_pieces", dict(ctx=[9000, 3000, 12000], k=[8, 8, 8], Hq=64, Hkv=8), 256, ANY),
    ("w5_many_pieces_kernel", dict(ctx=[9000, 3000, 12000], k=[8, 8, 8], Hq=64, Hkv=8), 256, None),
    # one-wave items, 20 and 8 pieces (51 KB per stream at most: fused by default)
    ("w1_mha", dict(ctx=[5000, 2000, 97], k=[4, 2, 0], Hq=4, Hkv=4), 256, None),
    # two and three waves, split and unsplit requests side by side (49 KB at most)
    ("w3_mixed", dict(ctx=[40, 6000, 700, 2100], k=[8, 1, 5, 3], Hq=32, Hkv=8), 512, None),
    ("w3_mixed_any", dict(ctx=[40, 6000, 700, 2100], k=[8, 1, 5, 3], Hq=32, Hkv=8), 512, ANY),
    # d = 64: 5 rows x 1877 pieces of 32 keys exceed the kernel's 32 KB of LDS,
    # so the separate combine kernel runs even with the limit lifted
    ("d64_fallback_kernel", dict(ctx=[60000], k=[4], Hq=1, Hkv=1, d=64), 32, ANY),
]


@pytest.fixture
def fuse_limit(monkeypatch):
    def set_limit(v):
        if v is None:
            monkeypatch.delenv("SPEC_FUSED_COMBINE_MAX_BYTES", raising=False)
        else:
            monkeypatch.setenv("SPEC_FUSED_COMBINE_MAX_BYTES", v)
    return set_limit


def _attention(pool, split_kv, junk_seed=None):
    b = DeviceBatch(pool, "cuda")
    v = Verifier(b, split_kv=split_kv)
    if junk_seed is not None:
        g = torch.Generator(device="cuda").manual_seed(junk_seed)
        v._ws.copy_(torch.randint(0, 256, v._ws.shape, dtype=torch.uint8, device="cuda", generator=g))
    v.run("attn")
    return v.results()["out"]


@pytest.mark.parametrize("name,kw,split,limit", CASES, ids=[c[0] for c in CASES])
def test_fused_combine_matches_oracle(gpu_lib, fuse_limit, name, kw, split, limit):
    fuse_limit(limit)
    seed = U.case_seed(name.replace("_kernel", "").replace("_any", ""))
    print(f"[case] {name} seed {seed} split_kv {split} fuse limit {limit}", flush=True)
    pool = U.custom_pool(seed=seed, **kw)
    out = _attention(pool, split)
    ref = U.oracle_attention_rows(pool, range(pool.batch))
    r = U.attention_ratios(out, pool, ref)
    print(f"{name} attention rows={r.size} worst={r.max():.3e}", flush=True)
    assert np.isfinite(r).all() and r.max() <= U.ATTN_RTOL, name
    # the same call over a workspace of random bytes: the arrival counters
    # start over on their first arrival, and the outputs are bit-identical
    for junk in (1, 2):
        again = _attention(pool, split, junk_seed=junk)
        assert np.array_equal(again.view(np.uint32), out.view(np.uint32)), (name, junk)


def test_fused_combine_repeated_calls(gpu_lib, fuse_limit):
    """Back-to-back calls on one workspace (the counters keep the previous
    call's values) give bit-identical outputs every time."""
    fuse_limit(ANY)
    name = "w5_repeat"
    pool = U.custom_pool(ctx=[7000, 150, 16000], k=[8, 3, 8], Hq=64, Hkv=8, seed=U.case_seed(name))
    print(f"[case] {name}", flush=True)
    b = DeviceBatch(pool, "cuda")
    v = Verifier(b, split_kv=384)
    outs = []
    for _ in range(4):
        b.out.fill_(float("nan"))
        v.run("attn")
        outs.append(v.results()["out"])
    for o in outs[1:]:
        assert np.array_equal(o.view(np.uint32), outs[0].view(np.uint32))
    ref = U.oracle_attention_rows(pool, range(pool.batch))
    assert U.attention_ratios(outs[0], pool, ref).max() <= U.ATTN_RTOL
