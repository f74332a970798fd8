"""GPU: verify calls captured into a HIP graph and replayed.

A captured call replays its kernel arguments, the call tag among them, so
the attention's tagged words (the split streams' arrival counters and the
item claim word) must be left ready for the same tag: each is reset by the
last work-group to use it in the call.  Every replay is checked bit for bit
against the eager call, with eager calls (new tags, same workspace) and
synchronisations between the replays.  The captured calls read the plan
staged at capture time, so the staging buffer is left untouched meanwhile.
"""
import numpy as np
import pytest
import torch

import parity_util as U
from paper_2505_17074_amd import binding as B
from paper_2505_17074_amd.batch import DeviceBatch

pytestmark = pytest.mark.gpu


def _outputs(b):
    torch.cuda.synchronize()
    return {"out": b.out.cpu().numpy(), "accepted_len": b.accepted_len.cpu().numpy(),
            "next_token": b.next_token.cpu().numpy(), "accepted_node": b.accepted_node.cpu().numpy()}


def _same(got, ref, what):
    assert np.array_equal(got["out"].view(np.uint32), ref["out"].view(np.uint32)), what
    for k in ("accepted_len", "next_token", "accepted_node"):
        assert np.array_equal(got[k], ref[k]), (what, k)


def _clear(b):
    b.out.fill_(float("nan"))
    b.accepted_len.fill_(-1)
    b.next_token.fill_(-1)
    b.accepted_node.fill_(-1)


@pytest.mark.parametrize("entry", ["verify", "verify_attn", "verify_noalloc"])
def test_graph_replays_match_eager_calls(gpu_lib, monkeypatch, entry):
    # split streams combined in the kernel (fused, the counters) and items
    # past a first round of two work-groups (the claim word)
    monkeypatch.setenv("SPEC_ATTN_FIRST_ROUND", "2")
    name = "graph_" + entry
    seed = U.case_seed(name)
    print(f"[case] {name} seed {seed}", flush=True)
    pool = U.custom_pool(ctx=[7000, 150, 16000, 900], k=[8, 3, 8, 5], Hq=32, Hkv=8, seed=seed)
    b = DeviceBatch(pool, "cuda")
    req, attn, acc = b.requests(), b.attn_args(384), b.accept_args()
    st, dev_bytes, host_bytes = B.spec_workspace_bytes(req, attn, acc)
    B.check(st, "spec_workspace_bytes")
    ws = torch.empty(dev_bytes + 256, dtype=torch.uint8, device="cuda")
    wsp = (ws.data_ptr() + 255) // 256 * 256
    staging = [torch.empty(max(host_bytes, 1), dtype=torch.uint8, pin_memory=True) for _ in range(2)]

    def call(stream, slot):
        h = stream.cuda_stream
        stg = staging[slot].data_ptr()
        if entry == "verify":
            return B.spec_verify(req, attn, acc, wsp, dev_bytes, stg, host_bytes, h)
        if entry == "verify_attn":
            return B.spec_verify_attn(req, attn, wsp, dev_bytes, stg, host_bytes, h)
        return B.spec_verify_noalloc(req, attn, acc, h)

    main = torch.cuda.current_stream()
    _clear(b)
    B.check(call(main, 0), entry)
    ref = _outputs(b)

    s = torch.cuda.Stream()
    s.wait_stream(main)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s, capture_error_mode="relaxed"):
        st = call(s, 1)
    B.check(st, entry + " (captured)")
    torch.cuda.synchronize()
    for rep in range(4):
        print(f"[case] {name} replay {rep}", flush=True)
        _clear(b)
        g.replay()
        got = _outputs(b)
        if entry == "verify_attn":
            assert np.array_equal(got["out"].view(np.uint32), ref["out"].view(np.uint32)), rep
        else:
            _same(got, ref, f"replay {rep}")
        if rep == 1:
            # an eager call between replays: a new tag on the same workspace
            _clear(b)
            B.check(call(main, 0), entry)
            got = _outputs(b)
            if entry == "verify_attn":
                assert np.array_equal(got["out"].view(np.uint32), ref["out"].view(np.uint32))
            else:
                _same(got, ref, "eager between replays")
    del g
