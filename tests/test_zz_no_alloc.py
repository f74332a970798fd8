"""spec_verify_noalloc (the entry point for callers that cannot allocate)
against spec_verify on the same inputs: two no-allocation calls enqueued
back to back on one stream with no synchronisation between them, the second
on a smaller step, and each compared bit for bit with spec_verify's outputs
(same kernels, same plan, so the same bits).  The first call splits long
requests, so its split partials and acceptance statistics live in the
library's static scratch; the second reuses that scratch."""
import numpy as np
import pytest
import torch

import parity_util as U
from paper_2505_17074_amd import binding as B
from paper_2505_17074_amd import workload as W
from paper_2505_17074_amd.batch import DeviceBatch, Verifier

pytestmark = pytest.mark.gpu


def _reference(pool):
    b = DeviceBatch(pool, "cuda")
    v = Verifier(b)
    v.run("verify")
    return v.results()


def _outputs(b):
    return {"out": b.out.cpu().numpy(), "accepted_len": b.accepted_len.cpu().numpy(),
            "next_token": b.next_token.cpu().numpy(), "accepted_node": b.accepted_node.cpu().numpy()}


@pytest.mark.parametrize("first,second", [
    ((3, 2), (1, 4)),        # long-context GQA (split partials) then a small MHA step
    ((2, 24), (4, 3)),       # ragged adaptive-k batch then a small token-tree step
])
def test_noalloc_matches_spec_verify(gpu_lib, first, second):
    print(f"[case] no-alloc: configs[{first[0]}] batch {first[1]} then configs[{second[0]}] batch {second[1]}",
          flush=True)
    pools = [W.make_pool(W.CONFIGS[i], 1, batch=n) for i, n in (first, second)]
    refs = [_reference(p) for p in pools]
    batches = [DeviceBatch(p, "cuda") for p in pools]
    for b in batches:
        b.out.fill_(float("nan"))
        for t in (b.accepted_len, b.next_token, b.accepted_node):
            t.fill_(-1)
    h = torch.cuda.current_stream().cuda_stream
    for b in batches:                  # back to back, no synchronisation in between
        st = B.spec_verify_noalloc(b.requests(), b.attn_args(), b.accept_args(), h)
        B.check(st, "spec_verify_noalloc")
    torch.cuda.synchronize()
    for pool, b, ref in zip(pools, batches, refs):
        got = _outputs(b)
        for key in ref:
            assert np.array_equal(np.asarray(got[key]).view(np.uint8), np.asarray(ref[key]).view(np.uint8)), key
        print(f"  {pool.cfg.name} b{pool.batch}: bit-identical to spec_verify, "
              f"accepted {got['accepted_len'].tolist()[:8]}", flush=True)


def test_noalloc_refuses_a_step_beyond_its_scratch(gpu_lib):
    print("[case] no-alloc: a step beyond the static scratch", flush=True)
    pool = U.custom_pool(ctx=[60000, 60000, 60000], k=[16, 16, 16], Hq=8, Hkv=2, V=64)
    b = DeviceBatch(pool, "cuda")
    b.out.fill_(float("nan"))
    h = torch.cuda.current_stream().cuda_stream
    st = B.spec_verify_noalloc(b.requests(), b.attn_args(split_kv=32), b.accept_args(), h)
    assert st == B.SPEC_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert torch.isnan(b.out).all()              # nothing was enqueued
