"""The LM head fused with acceptance (spec_lm_head_accept) on the GPU:
  * the logits it writes against the fp64 oracle, within the bound of fp32
    accumulation of exact bf16 x bf16 products, |err| <= K 2^-23 sum_k |h_k w_k|
    (twice the first-order bound K u sum |h w| with u = 2^-24), plus half an
    ulp of bf16 when they are stored in bf16: for |x| in [2^e, 2^(e+1)) the
    ulp is 2^(e-7), so half of it is at most 2^-8 |x|;
  * its acceptance outputs against spec_accept on the same stored logits and
    against the acceptance oracle on them: bit-exact except counted near
    ties (its normalisers come from tile statistics, summed in another order)."""
import numpy as np
import pytest
import torch

import parity_util as U
from oracle import lm_head_logits, verify_accept
from paper_2505_17074_amd import binding as B
from paper_2505_17074_amd import workload as W
from paper_2505_17074_amd.batch import DeviceBatch, LmHeadVerifier, pad_vocab_rows

pytestmark = pytest.mark.gpu


def _check_logits(pool, got, tag):
    ref = lm_head_logits(pool.hidden, pool.weight)
    absref = lm_head_logits(pool.hidden & np.uint16(0x7FFF), pool.weight & np.uint16(0x7FFF))
    K = pool.hidden.shape[1]
    bound = K * 2.0 ** -23 * absref
    if pool.logit_dtype == W.BF16:
        bound = bound + 2.0 ** -8 * np.abs(ref)
    g = W.as_f32(got, pool.logit_dtype).astype(np.float64)
    err = np.abs(g - ref)
    ratio = (err / np.maximum(bound, 1e-30)).max()
    print(f"{tag} logits {g.shape} max err {err.max():.3e}, worst err / bound {ratio:.3f}", flush=True)
    assert np.isfinite(g).all() and (err <= bound).all(), tag


def _check_accept(pool, lmv, got_logits, tag, rule=B.SPEC_TREE_INDEPENDENT):
    fused = lmv.results()
    # the unfused path on the same stored logits
    pool.target_logits = got_logits
    b = DeviceBatch(pool, "cuda")
    pad_vocab_rows(b)
    req, acc = b.requests(), b.accept_args(tree_rule=rule)
    st, dbytes, hbytes = B.spec_workspace_bytes(req, None, acc)
    B.check(st, "spec_workspace_bytes")
    ws = torch.empty(dbytes + 256, dtype=torch.uint8, device="cuda")
    staging = torch.empty(max(hbytes, 1), dtype=torch.uint8, pin_memory=True)
    B.check(B.spec_accept(req, acc, (ws.data_ptr() + 255) // 256 * 256, dbytes, staging.data_ptr(), hbytes,
                          torch.cuda.current_stream().cuda_stream), "spec_accept")
    torch.cuda.synchronize()
    unfused = {"accepted_len": b.accepted_len.cpu().numpy(), "next_token": b.next_token.cpu().numpy(),
               "accepted_node": b.accepted_node.cpu().numpy()}
    ref = verify_accept(got_logits, pool.draft_probs, pool.draft_tokens, pool.uniforms, pool.n_q,
                        dtype=pool.logit_dtype, tree_parent=pool.tree_parent, tree_parents=pool.tree_parents,
                        tree_rule="sequential" if rule == B.SPEC_TREE_SEQUENTIAL else "independent")
    bad, ties = U.compare_accept(fused, ref, pool)
    diff = [i for i in range(pool.batch) if not ref["near_tie"][i] and
            any(int(fused[k][i]) != int(unfused[k][i]) for k in ("accepted_len", "next_token", "accepted_node"))]
    print(f"{tag} accept B={pool.batch} mean_accepted={fused['accepted_len'].mean():.3f} near_ties={ties} "
          f"oracle mismatches={bad} unfused mismatches={diff}", flush=True)
    assert not bad and not diff, tag
    assert ties <= U.max_near_ties(pool.batch), (tag, ties)


CASES = [
    # (config, batch, hidden_dim, vocab override)
    ("tiny_f32", 4, 256, None),          # fp32 logits, 1024 entries
    ("mha7b_b32", 3, 64, 1000),          # vocabulary not a multiple of the 256-entry tile
    ("long_gqa_b8", 1, 128, 4099),       # bf16 logits, ragged vocabulary
    ("ragged_gqa_b128", 24, 256, 5000),  # 2 row tiles
    ("tree15_b64", 3, 512, 3000),        # token tree, every row's statistics from the GEMM
    ("mha7b_b32", 32, 4096, None),       # LLaMA-7B LM head at the full workload (160 rows)
    ("ragged_gqa_b128", 128, 4096, None),  # full workload: 716 rows, 192-row tiles
    ("tree15_b64", 64, 4096, None),      # full workload: 960 rows, 256-row tiles
    ("tiny_f32", 5, 96, 700),            # hidden width 96: a 64-k slice, then a 32-k tail slice
    ("mha7b_b32", 2, 32, 513),           # hidden width 32: the tail slice alone
]


@pytest.mark.parametrize("name,batch,K,V", CASES, ids=[f"{c[0]}-b{c[1]}-K{c[2]}" for c in CASES])
def test_lm_head_accept_against_the_oracle(gpu_lib, name, batch, K, V):
    cfg = W.CONFIG_BY_NAME[name]
    print(f"[case] LM head {name} batch {batch} K {K} V {V or cfg.vocab}, seed 1", flush=True)
    pool = W.make_lm_head_pool(cfg, 1, batch=batch, hidden_dim=K, vocab=V)
    lmv = LmHeadVerifier(pool, "cuda")
    lmv.batch.logits.fill_(float("nan"))
    lmv.run()
    got = lmv.logits()
    _check_logits(pool, got, name)
    _check_accept(pool, lmv, got, name)
    if pool.tree_parent is not None:
        lmv.acc.tree_rule = B.SPEC_TREE_SEQUENTIAL
        lmv.run()
        _check_accept(pool, lmv, lmv.logits(), name + "/seq", rule=B.SPEC_TREE_SEQUENTIAL)


@pytest.mark.parametrize("rule", [B.SPEC_TREE_INDEPENDENT, B.SPEC_TREE_SEQUENTIAL], ids=["independent", "sequential"])
def test_lm_head_per_request_trees(gpu_lib, rule):
    """Per-request trees through the LM head (the GEMM copies the node table
    to the device for the decision): requests alternate between the 15-node
    binary tree and a 15-node tree of another shape with the same seven
    nodes that have children (a chain 0..7 with one leaf under each of
    0..6), so the draft rows keep their layout; fp32 draft probabilities, so
    every draft token keeps a positive probability under its new parent."""
    cfg = W.CONFIG_BY_NAME["tree15_b64"]
    name = f"tree15_b64 per-request trees, rule {rule}"
    print(f"[case] LM head {name}, batch 8 K 256 V 3000, seed 1", flush=True)
    pool = W.make_lm_head_pool(cfg, 1, batch=8, hidden_dim=256, vocab=3000)
    binary = np.asarray(pool.tree_parent, np.int32)
    other = np.array([-1, 0, 1, 2, 3, 4, 5, 6, 0, 1, 2, 3, 4, 5, 6], np.int32)
    assert len(binary) == len(other) and set(binary[1:]) == set(other[1:])
    pool.tree_parents = [binary if i % 2 == 0 else other for i in range(pool.batch)]
    pool.tree_parent = None
    lmv = LmHeadVerifier(pool, "cuda")
    lmv.acc.tree_rule = rule
    lmv.batch.logits.fill_(float("nan"))
    lmv.run()
    got = lmv.logits()
    _check_logits(pool, got, name)
    _check_accept(pool, lmv, got, name, rule=rule)


def test_lm_head_long_context_vocabulary(gpu_lib):
    """The 64-head long-context workload's LM head: hidden size 8192,
    vocabulary 128256 (501 tiles), logits stored in bf16, 2 requests."""
    cfg = W.CONFIG_BY_NAME["long_gqa_b8"]
    print("[case] LM head long_gqa_b8 batch 2 K 8192 V 128256", flush=True)
    pool = W.make_lm_head_pool(cfg, 2, batch=2)
    lmv = LmHeadVerifier(pool, "cuda")
    lmv.run()
    got = lmv.logits()
    _check_logits(pool, got, "long")
    _check_accept(pool, lmv, got, "long")
