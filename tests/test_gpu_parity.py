"""GPU parity: the HIP verify path against the fp64 oracle on the same seeded inputs.

Every call goes through the C ABI (spec_verify / spec_verify_attn / spec_accept).
Tolerances are stated in parity_util: attention row-relative <= 2e-3;
accepted lengths, nodes and next tokens bit-exact except counted near ties.
"""
import itertools

import numpy as np
import pytest
import torch

import parity_util as U
from paper_2505_17074_amd import binding as B
from paper_2505_17074_amd import workload as W
from paper_2505_17074_amd.batch import DeviceBatch, Verifier

pytestmark = pytest.mark.gpu


def _say(msg):
    print(f"[case] {msg}", flush=True)


def _run(pool, which="verify", split_kv=0):
    b = DeviceBatch(pool, "cuda")
    v = Verifier(b, split_kv=split_kv)
    v.run(which)
    return v.results()


def _check(pool, res, attn_reqs=None, accept=True, tag=""):
    if attn_reqs is None:
        attn_reqs = range(pool.batch)
    if len(attn_reqs):
        ref = U.oracle_attention_rows(pool, attn_reqs)
        r = U.attention_ratios(res["out"], pool, ref)
        print(f"{tag} attention rows={r.size} worst={r.max():.3e} over1e-3={np.mean(r > 1e-3):.4f}", flush=True)
        assert np.isfinite(r).all() and r.max() <= U.ATTN_RTOL, tag
    if accept:
        ref = U.oracle_accept(pool)
        bad, ties = U.compare_accept(res, ref, pool)
        acc = res["accepted_len"]
        print(f"{tag} accept B={pool.batch} mean_accepted={acc.mean():.3f} near_ties={ties} mismatches={bad}",
              flush=True)
        assert not bad, (tag, bad)
        assert ties <= U.max_near_ties(pool.batch), (tag, ties)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_tiny_f32(gpu_lib, seed):
    _say(f"tiny_f32 seed={seed}")
    pool = W.make_pool(W.CONFIGS[0], seed)
    _check(pool, _run(pool), tag=f"tiny_f32/{seed}")


REDUCED = {1: 6, 2: 24, 3: 2, 4: 6}


@pytest.mark.parametrize("idx,seed", [(i, s) for i in (1, 2, 3, 4) for s in (0, 1)])
def test_reduced_batches(gpu_lib, idx, seed):
    cfg = W.CONFIGS[idx]
    _say(f"{cfg.name} batch={REDUCED[idx]} seed={seed}")
    pool = W.make_pool(cfg, seed, batch=REDUCED[idx])
    _check(pool, _run(pool), tag=f"{cfg.name}/b{REDUCED[idx]}/{seed}")


@pytest.mark.parametrize("idx", [1, 2, 3, 4])
def test_full_size_every_request(gpu_lib, idx):
    """Full-size workloads in the benchmark's launch configuration: every
    request's attention against the oracle, element by element, and the
    acceptance of every request.  The output and the workspace start as NaN
    bytes, so a lost or misrouted work item would leave rows unwritten or
    filled from stale scratch; three runs must agree bit for bit (each row
    has one producer and the combine merges partials in a fixed order)."""
    cfg = W.CONFIGS[idx]
    _say(f"{cfg.name} full size, seed 0")
    pool = U.full_pool(idx)
    b = DeviceBatch(pool, "cuda")
    v = Verifier(b)
    outs = []
    for rep in range(3):
        v._ws.fill_(255)
        b.out.fill_(float("nan"))
        b.accepted_len.fill_(-1)
        b.next_token.fill_(-1)
        v.run("verify")
        outs.append(v.results())
    for o in outs[1:]:
        for key in o:
            assert np.array_equal(np.asarray(o[key]).view(np.uint8), np.asarray(outs[0][key]).view(np.uint8)), key
    _check(pool, outs[0], tag=f"{cfg.name}/full")
    del b, v
    torch.cuda.empty_cache()


ODD_VOCAB = [
    ("vocab_odd_f32", dict(ctx=[1, 2, 3], k=[3, 0, 5], V=4099)),
    ("vocab_odd_bf16", dict(ctx=[1, 2, 3], k=[3, 0, 5], V=8199, logit=W.BF16)),
    ("vocab_3", dict(ctx=[1, 2, 3, 4], k=[1, 2, 3, 16], V=3)),
    ("plain_decode_only", dict(ctx=[5] * 9, k=[0] * 9, V=1000)),
]


@pytest.mark.parametrize("name,kw", ODD_VOCAB, ids=[e[0] for e in ODD_VOCAB])
def test_accept_padded_rows(gpu_lib, name, kw):
    """Vocabularies that are not a multiple of a 16-byte load: the rows are
    stored with a padded stride (NaN in the padding, which must never be
    read), so one vector load straddles the vocabulary's end."""
    seed = U.case_seed(name)
    _say(f"{name} padded rows, seed {seed}")
    pool = U.custom_pool(**kw, seed=seed)
    b = DeviceBatch(pool, "cuda")
    V = pool.vocab
    vec = 8 if pool.logit_dtype == W.BF16 else 4
    Vp = -(-V // vec) * vec
    for attr in ("logits", "probs"):
        t = getattr(b, attr)
        if t.numel():
            pad = torch.full((t.shape[0], Vp + vec), float("nan"), dtype=t.dtype, device=t.device)
            pad[:, :V] = t
            setattr(b, attr, pad[:, :V])
    v = Verifier(b)
    v.run("accept")
    _check(pool, v.results(), attn_reqs=[], tag=name)


def test_split_invariance(gpu_lib):
    pool = W.make_pool(W.CONFIGS[1], 3, batch=4)
    outs = {}
    for split in (32, 96, 512, 0, 1 << 16):
        _say(f"split_kv={split}")
        res = _run(pool, split_kv=split)
        _check(pool, res, accept=(split == 0), tag=f"split{split}")
        outs[split] = res
    base = outs[0]
    for split, res in outs.items():
        np.testing.assert_allclose(res["out"], base["out"], rtol=0, atol=5e-3 * np.abs(base["out"]).max())


@pytest.mark.parametrize("cfg_idx,batch", [(2, 24), (4, 6)])
def test_pageable_staging_matches_pinned(gpu_lib, cfg_idx, batch):
    """A staging buffer in pageable host memory has no device mapping, so the
    plan is copied into the workspace before the kernels (instead of being
    read where it was staged): the outputs must be bit-identical.  The ragged
    batch splits requests, so the combine's copies are exercised too."""
    cfg = W.CONFIGS[cfg_idx]
    _say(f"{cfg.name} b{batch}: pageable staging")
    pool = W.make_pool(cfg, 2, batch=batch)
    b = DeviceBatch(pool, "cuda")
    v = Verifier(b)
    v.run("verify")
    ref = v.results()
    b.out.fill_(float("nan"))
    b.accepted_len.fill_(-1)
    b.next_token.fill_(-1)
    staging = np.zeros(v.staging_bytes + 64, np.uint8)          # pageable
    h = torch.cuda.current_stream().cuda_stream
    B.check(B.spec_verify(v.req, v.attn, v.acc, v.ws_ptr, v.ws_bytes, staging.ctypes.data, v.staging_bytes, h),
            "spec_verify")
    got = v.results()
    for key in ref:
        assert np.array_equal(np.asarray(got[key]).view(np.uint8), np.asarray(ref[key]).view(np.uint8)), key


@pytest.mark.parametrize("batch", [40, 96])
def test_many_split_requests(gpu_lib, batch):
    """128-key pieces split nearly every request (40 of 40, 93 of 96): many
    split requests, each with many pieces, through the split kernel's copies
    of the plan and the combine."""
    _say(f"ragged b{batch} split_kv=128")
    pool = W.make_pool(W.CONFIGS[2], 4, batch=batch)
    split = int(((pool.ctx_len.astype(np.int64) + pool.n_q) > 128).sum())
    assert (split <= 64) == (batch == 40), split
    res = _run(pool, split_kv=128)
    B = pool.batch
    _check(pool, res, attn_reqs=sorted({0, 1, B // 2, B - 2, B - 1}), tag=f"b{batch}/split128")


def test_deterministic(gpu_lib):
    _say("determinism ragged_gqa b32")
    pool = W.make_pool(W.CONFIGS[2], 5, batch=32)
    b = DeviceBatch(pool, "cuda")
    v = Verifier(b)
    v.run()
    first = v.results()
    for _ in range(3):
        v.run()
    second = v.results()
    for key in first:
        assert np.array_equal(first[key], second[key]), key


EDGE = [
    ("ctx_edges_k0_k16", dict(ctx=[0, 1, 31, 32, 33, 100], k=[0, 1, 16, 4, 0, 7])),
    ("d64_mha", dict(ctx=[17, 300, 64], k=[3, 0, 8], Hq=4, Hkv=4, d=64)),
    ("f32_valu_gqa_d128", dict(ctx=[5, 130, 70], k=[2, 6, 0], Hq=8, Hkv=2, d=128, qkv=W.F32)),
    ("f32_valu_d64", dict(ctx=[200, 0], k=[16, 3], Hq=2, Hkv=1, d=64, qkv=W.F32)),
    ("tree_nonbinary", dict(ctx=[0, 50, 300], tree_parent=[-1, 0, 0, 0, 1, 1, 2, 4, 4, 7])),
    ("wide_group_split", dict(ctx=[90, 40], k=[16, 9], Hq=32, Hkv=2)),
    ("vocab_5000_bf16_logits", dict(ctx=[10, 20, 30, 40], k=[4, 3, 2, 1], V=5000, logit=W.BF16)),
    ("vocab_tail_f32", dict(ctx=[10, 20], k=[4, 8], V=4100)),
    ("long_single", dict(ctx=[20000], k=[5])),
    # bf16 kernel widths: at most 32 rows per item -> two waves (one split
    # request so the combine runs too), at d = 128 and d = 64; 36 rows -> three
    ("gqa_two_waves_d128", dict(ctx=[300, 1200, 40, 5000], k=[5, 7, 3, 7], Hq=8, Hkv=2)),
    ("gqa_two_waves_d64", dict(ctx=[100, 2500], k=[7, 2], Hq=8, Hkv=2, d=64)),
    ("gqa_three_waves_short", dict(ctx=[33, 65, 0], k=[8, 1, 2], Hq=8, Hkv=2)),
    # uneven wave splits of a tile's transfers (the first waves issue one
    # more than the rest, each waits on its own count): 3 and 5 waves at
    # d = 64 (8 transfers a tile) and 5 waves at d = 128 (16), ragged
    # contexts and a split request
    ("gqa_three_waves_d64", dict(ctx=[1000, 7, 6100, 95], k=[8, 3, 8, 5], Hq=8, Hkv=2, d=64)),
    ("gqa_five_waves_d64", dict(ctx=[2500, 41, 9000], k=[8, 8, 2], Hq=16, Hkv=2, d=64)),
    ("gqa_five_waves_d128", dict(ctx=[3001, 100, 12000, 0], k=[8, 8, 3, 8], Hq=16, Hkv=2)),
]


@pytest.mark.parametrize("name,kw", EDGE, ids=[e[0] for e in EDGE])
def test_edge_cases(gpu_lib, name, kw):
    seed = U.case_seed(name)
    _say(f"{name} seed {seed}")
    pool = U.custom_pool(**kw, seed=seed)
    _check(pool, _run(pool), tag=name)


def test_custom_scale_and_strided_query(gpu_lib):
    _say("custom scale, head-major query layout")
    pool = U.custom_pool(ctx=[40, 77], k=[3, 5], Hq=8, Hkv=2)
    b = DeviceBatch(pool, "cuda")
    # store Q head-major ([Hq, Nq, d]) and pass its strides
    qhm = b.q.permute(1, 0, 2).contiguous()
    b.q = qhm.permute(1, 0, 2)
    v = Verifier(b)
    v.attn.q = b.q.data_ptr()
    v.attn.q_stride_tok, v.attn.q_stride_head = b.q.stride(0), b.q.stride(1)
    v.attn.scale = 0.05
    v.run("attn")
    res = v.results()
    from oracle import verify_attention
    ref = verify_attention(pool.q, pool.k, pool.v, pool.ctx_len, pool.n_q, 2, dtype=pool.qkv_dtype, scale=0.05)
    r = np.abs(res["out"] - ref).max(-1) / np.abs(ref).max(-1)
    assert r.max() <= U.ATTN_RTOL


def test_p_equals_q_accepts_every_draft(gpu_lib):
    _say("p == q")
    pool = U.custom_pool(ctx=[3] * 8, k=[1, 2, 3, 4, 5, 6, 7, 8], V=2048)
    # draft rows := the target softmax (fp32), uniforms kept below 0.99
    lg = pool.target_logits.astype(np.float64)
    q0, d0 = pool.q_start, pool.d_start
    for i in range(pool.batch):
        for j in range(int(pool.draft_len[i])):
            row = lg[q0[i] + j]
            e = np.exp(row - row.max())
            pool.draft_probs[d0[i] + j] = (e / e.sum()).astype(np.float32)
    pool.uniforms[:] = np.minimum(pool.uniforms, np.float32(0.99))
    res = _run(pool, "accept")
    assert np.array_equal(res["accepted_len"], pool.draft_len)


def test_hand_packed_two_requests(gpu_lib):
    """The two-request batch worked by hand (parity_util.hand_packed_case)
    through spec_accept: the kernels' batch indexing against hand values."""
    _say("hand-packed two requests")
    inp, expect = U.hand_packed_case()
    pool = U.custom_pool(ctx=inp["ctx"], k=inp["draft_len"], Hq=1, Hkv=1, d=64, V=4)
    for key in ("target_logits", "draft_probs", "draft_tokens", "uniforms"):
        getattr(pool, key)[:] = inp[key]
    res = _run(pool, "accept")
    assert res["accepted_len"].tolist() == expect["accepted_len"]
    assert res["next_token"].tolist() == expect["next_token"]


@pytest.mark.parametrize("logit", [W.F32, W.BF16])
def test_accept_edge_rows(gpu_lib, logit):
    """The oracle's special cases through the kernels, bit-exact:
      0  p(x) = 0 at a draft token (logit -1e30: zero in fp32 and fp64) with
         u = 0: 0 * q < 0 fails, rejected at once;
      1  one-hot draft row at a token the target gives p = 0: rejected, the
         residual is p itself;
      2  one-hot draft row at a token with p > 0 and u = 0: accepted;
      3  draft row stored as 1.1 p with u = 0.95: rejected, and
         max(0, p - 1.1 p) has zero mass, so the final token falls back to p;
      4  u = 0 on every test and on the final sample: every draft accepted,
         the extra token is the smallest id with positive weight;
      5  u = 0 on the tests but p(x) = 0 at the second draft: a = 1;
      6  p(x) = 0 at draft 0 and u = 0 on the final sample: the smallest id
         with positive residual weight."""
    _say(f"accept edge rows, logits {logit}")
    V = 1000
    pool = U.custom_pool(ctx=[3, 4, 5, 6, 7, 8, 9], k=[3, 2, 2, 3, 4, 2, 2], V=V, logit=logit,
                         seed=U.case_seed(f"edge_rows_{logit}"))
    q0, d0 = pool.q_start, pool.d_start
    tl = W.as_f32(pool.target_logits, logit).astype(np.float32).copy()
    qp = W.as_f32(pool.draft_probs, logit).astype(np.float32).copy()
    tok, u = pool.draft_tokens, pool.uniforms
    NEG = np.float32(-1e30)

    def tokidx(i, j):                  # request i's draft j (0-based) in the packed token array
        return int(q0[i]) - i + j

    # 0: p(x) = 0 at draft 0, u = 0
    tl[q0[0], tok[tokidx(0, 0)]] = NEG
    u[q0[0]] = 0.0
    # 1: one-hot q at x, p(x) = 0
    x = int(tok[tokidx(1, 0)])
    qp[d0[1]] = 0.0
    qp[d0[1], x] = 1.0
    tl[q0[1], x] = NEG
    # 2: one-hot q at x, p(x) > 0, u = 0
    x = int(tok[tokidx(2, 0)])
    qp[d0[2]] = 0.0
    qp[d0[2], x] = 1.0
    u[q0[2]] = 0.0
    # 3: q = 1.1 p (p from the stored logits), u = 0.95 at draft 0
    row = tl[q0[3]].astype(np.float64)
    e = np.exp(row - row.max())
    qp[d0[3]] = (1.1 * e / e.sum()).astype(np.float32)
    u[q0[3]] = 0.95
    # 4: u = 0 everywhere
    u[q0[4]:q0[5]] = 0.0
    # 5: u = 0 on the tests, p(x) = 0 at draft 1
    u[q0[5]:q0[5] + 2] = 0.0
    tl[q0[5] + 1, tok[tokidx(5, 1)]] = NEG
    # 6: p(x) = 0 at draft 0, u = 0 on the final sample
    tl[q0[6], tok[tokidx(6, 0)]] = NEG
    u[q0[6] + 2] = 0.0
    pool.target_logits[:] = W.storage(tl, logit)
    pool.draft_probs[:] = W.storage(qp, logit)
    ref = U.oracle_accept(pool)
    # the constructed outcomes, from the rule itself
    a = ref["accepted_len"].tolist()
    assert a[0] == 0 and a[1] == 0 and a[2] >= 1 and a[3] == 0 and a[4] == 4 and a[5] == 1 and a[6] == 0, a
    assert ref["next_token"][4] == 0
    res = _run(pool, "accept")
    for key in ("accepted_len", "next_token", "accepted_node"):
        assert res[key].tolist() == ref[key].tolist(), (key, res[key], ref[key])


@pytest.mark.parametrize("V,logit", [(1000, W.F32), (32000, W.F32), (8200, W.BF16)])
def test_path_tree_equals_chain(gpu_lib, V, logit):
    """A tree whose parent array is a path (parent(n) = n - 1) is the chain:
    bit-identical accepted lengths and next tokens, and the deepest accepted
    node is the accepted length.  Under the independent tree rule the last
    node's row is a leaf's, whose chunk statistics the decision kernel takes
    itself, with the row-statistics kernel's arithmetic."""
    import copy
    _say(f"path tree == chain, V={V}")
    K = 6
    # target close to the draft (sigma 0.15): about half the requests accept
    # every draft and sample from the last (leaf) row
    chain = U.custom_pool(ctx=[3, 40, 7, 90, 1, 0, 12, 33] * 2, k=[K] * 16, V=V, logit=logit, seed=V, sigma=0.15)
    tree = copy.copy(chain)
    tree.tree_parent = np.arange(-1, K, dtype=np.int32)
    a = _run(chain, "accept")
    b = _run(tree, "accept")
    assert np.array_equal(a["accepted_len"], b["accepted_len"])
    assert np.array_equal(a["next_token"], b["next_token"])
    assert np.array_equal(b["accepted_node"], b["accepted_len"])
    _check(chain, a, attn_reqs=[], tag="chain")


def _cells(breaks):
    b = sorted(set([0.0, 1.0] + [float(x) for x in breaks if 0.0 < x < 1.0]))
    return [((lo + hi) / 2.0, hi - lo) for lo, hi in zip(b[:-1], b[1:])]


def test_emitted_token_distribution_exact_on_gpu(gpu_lib):
    """The vocab-8 identity, black-box through the GPU kernels: one request per
    uniform cell; summing cell probabilities by the GPU's outcomes must give
    the target distribution exactly (every midpoint is far from a boundary)."""
    _say("vocab-8 enumeration through the GPU")
    V = 8
    rng = np.random.default_rng(17)
    p0 = rng.random(V) ** 2 + 0.01
    p0 /= p0.sum()
    p1 = rng.random(V) + 0.01
    p1 /= p1.sum()
    q0 = rng.random(V) + 0.01
    q0 /= q0.sum()
    q0 = q0.astype(np.float32).astype(np.float64)
    q0 /= q0.sum()
    q0 = q0.astype(np.float32)
    qd = q0.astype(np.float64)
    res = np.maximum(0, p0 - qd)
    fin = []
    for w in (res, p1):
        fin.extend(np.cumsum(w) / w.sum())
    cases = []
    for x in range(V):
        for (u0, l0), (u1, l1) in itertools.product(_cells([min(1.0, p0[x] / qd[x])]), _cells(fin)):
            cases.append((x, np.float32(u0), np.float32(u1), qd[x] * l0 * l1))
    n = len(cases)
    pool = U.custom_pool(ctx=[0] * n, k=[1] * n, Hq=1, Hkv=1, d=64, V=V)
    pool.target_logits[:] = np.tile(np.log(np.stack([p0, p1])).astype(np.float32), (n, 1))
    pool.draft_probs[:] = np.tile(q0[None], (n, 1))
    pool.draft_tokens[:] = [c[0] for c in cases]
    pool.uniforms[:] = np.array([[c[1], c[2]] for c in cases], np.float32).ravel()
    out = _run(pool, "accept")
    dist = np.zeros(V)
    for i, (x, _, _, w) in enumerate(cases):
        y = x if out["accepted_len"][i] == 1 else out["next_token"][i]
        dist[y] += w
    np.testing.assert_allclose(dist, p0, rtol=0, atol=1e-6)


def test_statistical_acceptance_monte_carlo(gpu_lib):
    """2^20 independent verify rounds through the GPU kernels at vocabulary 8,
    k = 4, with target and draft rows that do not depend on the prefix:
      * the mean accepted length matches sum_{j=1..k} prod_{t<j} alpha_t,
        alpha_t = sum_x min(p_t(x), q_t(x)) (Sec. 4.3: n*A accepted drafts
        per round), within 5 standard errors;
      * the first emitted token (the first draft if accepted, else the final
        sample) follows p_0: chi-square p-value above 1e-6."""
    from scipy import stats
    _say("Monte Carlo acceptance, vocab 8, k 4, 2^20 rounds")
    V, k, B, rounds = 8, 4, 1 << 16, 16
    rng = np.random.default_rng(23)
    logits = np.log(rng.dirichlet(np.ones(V), size=k + 1)).astype(np.float32)
    Q = rng.dirichlet(np.ones(V), size=k).astype(np.float32)
    pool = U.custom_pool(ctx=[0] * B, k=[k] * B, Hq=1, Hkv=1, d=64, V=V)
    pool.target_logits[:] = np.tile(logits, (B, 1))
    pool.draft_probs[:] = np.tile(Q, (B, 1))
    b = DeviceBatch(pool, "cuda")
    v = Verifier(b, ring=2, event_every=1)
    # the distributions the kernels see: p from the stored logits, q as stored
    P = np.exp(logits.astype(np.float64))
    P /= P.sum(1, keepdims=True)
    Qd = Q.astype(np.float64)
    alpha = np.minimum(P[:k], Qd).sum(1)
    expect = sum(np.prod(alpha[:j]) for j in range(1, k + 1))
    acc, first = [], []
    for _ in range(rounds):
        toks = np.stack([rng.choice(V, size=B, p=Qd[t] / Qd[t].sum()) for t in range(k)], 1).astype(np.int32)
        u = (rng.integers(0, 1 << 24, size=(B, k + 1)) * 2.0 ** -24).astype(np.float32)
        b.tokens.copy_(torch.from_numpy(toks.ravel()))
        b.uniforms.copy_(torch.from_numpy(u.ravel()))
        v.run("accept")
        res = v.results()
        a = res["accepted_len"].astype(np.int64)
        assert ((a >= 0) & (a <= k)).all()
        acc.append(a)
        first.append(np.where(a >= 1, toks[:, 0], res["next_token"]))
    a, y = np.concatenate(acc), np.concatenate(first)
    se = a.std() / np.sqrt(a.size)
    print(f"mean accepted {a.mean():.5f} closed form {expect:.5f} (se {se:.5f})", flush=True)
    assert abs(a.mean() - expect) < 5 * se
    counts = np.bincount(y, minlength=V)
    chi2, pval = stats.chisquare(counts, P[0] * y.size)
    print(f"first token chi2 {chi2:.2f} p-value {pval:.3g}", flush=True)
    assert pval > 1e-6
