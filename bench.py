"""Benchmark of the batched speculative-decoding verify step on one MI355X.

A step is one spec_verify call over one batch: host plan (staged), split-KV
verify attention (+ combine), acceptance and the final sample -- every row of
the hot path -- over inputs already resident in HBM.  Prints ONE JSON line.

  python bench.py [--steps K] [--warmup W] [--workload NAME] [--only] [--no-cpu] [--no-sched]

The headline is the largest single-GPU workload (128 ragged GQA requests);
the other workloads are measured the same way in the same run and reported
under "workloads".
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "verified tokens/s per verify step; achieved HBM GB/s vs MI355X peak"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, vendor figure
EVENT_EVERY = 4                # timed steps per pair of kernel-timing events
MFMA_BF16_PEAK = 2.5e15         # MI355X dense bf16 matrix FLOP/s, vendor figure


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=HEADLINE,
                    help="the headline workload (default: the largest that fits one GPU)")
    ap.add_argument("--only", action="store_true", help="measure the headline workload only (profiler runs)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-sched", action="store_true",
                    help="skip the scheduler's closed loop (thousands of small launches; for profiler runs)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-lm-head", action="store_true", help="skip the fused LM-head figures")
    ap.add_argument("--settle", type=float, default=0.3, metavar="SECONDS",
                    help="untimed steps for this long before the warm-up steps, while the clocks ramp")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="only copy BYTES device-to-device three times (the calibration run for the "
                         "rocprofv3 FETCH_SIZE / WRITE_SIZE counters) and exit")
    return ap.parse_args()


def copy_probe(nbytes: int) -> None:
    """A plain device copy of known size: reads and writes nbytes per launch."""
    import torch
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
    dst = torch.empty_like(src)
    src.fill_(1)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": nbytes, "launches": 3}), flush=True)


def stream_ceilings_gbs(dev, nbytes: int = 2 << 30, reps: int = 5):
    """Measured stream rates over nbytes, far beyond the 256 MB Infinity
    Cache, reported beside the vendor peak: the library's plain read probe
    (spec_stream_read_probe, the best of a few grid sizes; bytes read per
    second -- the attention kernel is read-dominated) and a device copy
    (bytes read plus written per second)."""
    import torch
    from paper_2505_17074_amd import binding as B
    src = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    src.fill_(1)
    out = torch.empty(1 << 16, dtype=torch.int32, device=dev)
    h = torch.cuda.current_stream(dev).cuda_stream
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def rate(fn, moved):
        fn()
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return moved / (e0.elapsed_time(e1) * 1e-3 / reps) / 1e9

    def probe(blocks):
        B.check(B.spec_stream_read_probe(src.data_ptr(), nbytes, out.data_ptr(), blocks, h), "spec_stream_read_probe")

    read = max(rate(lambda: probe(g), nbytes) for g in (512, 2048, 8192, 32768, 65536))
    dst = torch.empty_like(src)
    copy = rate(lambda: dst.copy_(src), 2 * nbytes)
    del src, dst, out
    torch.cuda.empty_cache()
    return read, copy


class CacheFlush:
    """Leaves the L2s and the 256 MB Infinity Cache holding clean lines of a
    1 GiB scratch buffer: a write of it, then a read (both untimed).  A write
    alone would leave dirty lines whose write-back lands in the next timed
    call."""

    def __init__(self, dev):
        import torch
        self.buf = torch.empty(1 << 28, dtype=torch.float32, device=dev)
        self.sink = torch.empty((), dtype=torch.float32, device=dev)

    def __call__(self):
        import torch
        self.buf.fill_(1.0)
        torch.sum(self.buf, dim=(0,), out=self.sink)


def pct(xs, q):
    import numpy as np
    return float(np.percentile(np.asarray(xs, dtype=np.float64), q))


def scheduler_closed_loop(dev, seed: int) -> dict:
    """The LAPS-SD scheduler driven by the verify step's own accepted counts:
    50 requests' per-round accepted counts from the library's acceptance
    kernels (one batched spec_accept per round index), then every policy on
    the one-request-at-a-time server model, and the native scheduler's cost
    per decision."""
    from paper_2505_17074_amd import closed_loop as CL
    from paper_2505_17074_amd.scheduler import simulate
    swap = CL.measure_swap(dev)
    verify = CL.measure_verify(dev)
    cfg = CL.LoopConfig(swap_us_per_token=swap["us_per_token"], verify_us=verify)
    wl = CL.make_workload(cfg, seed)
    t0 = time.perf_counter()
    traces = CL.gpu_traces(cfg, wl, seed, device=dev)
    t_traces = time.perf_counter() - t0
    reqs = CL.requests_from(cfg, wl, traces)
    params = CL.default_params(cfg)
    res = CL.evaluate(reqs, params)
    lat = {pol: r["avg_latency_ms"] for pol, r in res.items()}
    reps, t0 = 20, time.perf_counter()
    for _ in range(reps):
        o = simulate(reqs, "laps_sd", params, log=False)
    dec_us = (time.perf_counter() - t0) / reps / o["n_rounds"] * 1e6
    return {"workload": f"{cfg.requests} requests, draft {cfg.draft}, output lengths log-normal (median "
                        f"{cfg.out_median}), predicted with log-normal error sigma {cfg.pred_sigma}, per-request "
                        f"acceptance from target noise sigma in {list(cfg.sigma)}; rounds "
                        f"{cfg.draft} x {cfg.t_ssm_us} + {cfg.t_llm_us} us + the measured verify kernels (32 layers' "
                        f"attention + acceptance) at the request's context; KV swap {cfg.swap_us_per_token} us/token",
            "verify_us_by_context": verify,
            "rounds_traced": int(traces.shape[1]), "trace_s": t_traces,
            "mean_tokens_per_round": float((traces + 1).mean()),
            "avg_latency_ms": lat,
            "switches": {pol: r["switches"] for pol, r in res.items()},
            "laps_sd_perceptible": res["laps_sd"]["perceptible"],
            "native_decision_us": dec_us,
            "kv_swap": {"d2h_GBs": swap["d2h_GBs"], "h2d_GBs": swap["h2d_GBs"],
                        "us_per_token_measured": swap["us_per_token"],
                        "bytes_per_token": CL.KV_BYTES_PER_TOKEN}}


def scheduler_oracle_decision_us(dev, seed: int) -> float:
    """The scheduler oracle's cost per decision on the same workload, with
    host-drawn traces of the same shape (the cost does not depend on the
    accepted counts' source)."""
    from oracle.scheduler import Params, Request, simulate
    from paper_2505_17074_amd import closed_loop as CL
    import numpy as np
    cfg = CL.LoopConfig()
    wl = CL.make_workload(cfg, seed)
    rng = np.random.default_rng(seed)
    traces = rng.binomial(cfg.draft, rng.uniform(0.2, 0.8, size=(cfg.requests, 1)),
                          size=(cfg.requests, int(wl.out_len.max())))
    reqs = [Request(r.arrival, r.prompt, r.out_len, r.pred_len, r.draft, r.round_us, list(r.accepted))
            for r in CL.requests_from(cfg, wl, traces)]
    p = CL.default_params(cfg)
    t0 = time.perf_counter()
    o = simulate(reqs, "laps_sd", Params(p.K, p.S1_up, p.M, p.gamma, p.delta, p.t_ssm, p.t_llm, p.swap_us_per_token))
    return (time.perf_counter() - t0) / len(o["log"]) * 1e6


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


# The sources the attention kernels are compiled from (the kernels and the two
# headers they include): counter figures taken on other sources are stale.
ATTN_SOURCES = ("attention.hip", "sv_attn.h", "sv_common.h")


def kernel_source_digest() -> str:
    h = hashlib.sha256()
    for name in ATTN_SOURCES:
        with open(os.path.join(ROOT, "paper_2505_17074_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload: str):
    """HBM bytes per call of the attention kernels (split-KV kernel and split
    combine) from the committed rocprofv3 counter summary, if it was taken on
    the current kernel source."""
    path = os.path.join(ROOT, "profiles", f"attn_split_{workload}_traffic.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    sha = re.search(r"kernel_source_sha256_16:\s*([0-9a-f]+)", text)
    val = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not sha or not val or sha.group(1) != kernel_source_digest():
        return None
    return float(val.group(1))


def cpu_baseline(pool, budget_s: float):
    """The fp64 oracle (untuned) on a bounded sample of the same requests:
    requests in order, wrapping around the batch, until about budget_s of host
    work (so small batches are timed over several passes)."""
    import numpy as np
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([d.get("num_threads", 1) for d in threadpool_info()] or [1])
    except Exception:                                   # pragma: no cover
        threads = 1
    q0, kv0, n_q = pool.q_start, pool.kv_start, pool.n_q
    done_tokens, t_used, m = 0, 0.0, 0
    while t_used < budget_s:
        i = m % pool.batch
        n, c = int(n_q[i]), int(pool.ctx_len[i])
        t0 = time.perf_counter()
        oracle.verify_attention(pool.q[q0[i]:q0[i] + n], pool.k[kv0[i]:kv0[i + 1]], pool.v[kv0[i]:kv0[i + 1]],
                                [c], [n], pool.num_kv_heads, dtype=pool.qkv_dtype, tree_parent=pool.parents_of(i))
        oracle.verify_accept(pool.target_logits[q0[i]:q0[i] + n], pool.draft_probs[pool.d_start[i]:pool.d_start[i + 1]],
                             pool.draft_tokens[q0[i] - i:q0[i] - i + n - 1], pool.uniforms[q0[i]:q0[i] + n], [n],
                             dtype=pool.logit_dtype, tree_parent=pool.parents_of(i))
        t_used += time.perf_counter() - t0
        done_tokens += n
        m += 1
    try:
        avail = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):                   # pragma: no cover
        avail = os.cpu_count() or 1
    return {"value": done_tokens / t_used, "unit": "verified tokens/s", "cores": int(threads),
            "cores_available": int(avail), "blas_threads": int(threads), "cpu_model": cpu_model(),
            "kind": "oracle",
            "sample": f"{m} request verifications ({m / pool.batch:.2f} passes over the {pool.batch} requests, "
                      f"{done_tokens} verify tokens), attention + acceptance in fp64 NumPy, {t_used:.1f} s"}


def lm_head_figures(name: str, seed: int, dev, flush, reps: int = 10) -> dict:
    """The LM head fused with acceptance (spec_lm_head_accept) on the
    workload's verify positions: the GEMM's time (events around its kernel,
    after a cache flush), its MFMA and HBM rooflines, torch's bf16 linear
    (hipBLASLt) on the same tensors as a reference point, and the fused
    acceptance (the decision on the GEMM's tile statistics) beside the
    unfused one (row pass + decision) on the same logits."""
    import numpy as np
    import torch
    from paper_2505_17074_amd import binding as B
    from paper_2505_17074_amd import workload as W
    from paper_2505_17074_amd.batch import LmHeadVerifier
    print(f"[bench] {name}: LM head", file=sys.stderr, flush=True)
    pool = W.make_lm_head_pool(W.CONFIG_BY_NAME[name], seed)
    lmv = LmHeadVerifier(pool, dev)
    M, K = pool.hidden.shape
    V = pool.vocab
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
    for e in ev:
        e.record()
    torch.cuda.synchronize()
    lmv.lm.event_begin, lmv.lm.event_end = ev[0].cuda_event, ev[1].cuda_event
    lmv.acc.event_begin, lmv.acc.event_end = ev[2].cuda_event, ev[3].cuda_event
    g, a, t = [], [], []
    for rep in range(reps + 2):
        flush()
        lmv.run()
        torch.cuda.synchronize()
        g.append(ev[0].elapsed_time(ev[1]) * 1e3)
        a.append(ev[2].elapsed_time(ev[3]) * 1e3)
    for rep in range(reps + 2):
        flush()
        ev[4].record()
        y = torch.nn.functional.linear(lmv.hidden, lmv.weight)
        ev[5].record()
        torch.cuda.synchronize()
        t.append(ev[4].elapsed_time(ev[5]) * 1e3)
    del y
    # the unfused acceptance on the logits the GEMM wrote
    b = lmv.batch
    req, acc = b.requests(), b.accept_args()
    st, db, hb = B.spec_workspace_bytes(req, None, acc)
    B.check(st, "spec_workspace_bytes")
    ws = torch.empty(db + 256, dtype=torch.uint8, device=dev)
    stg = torch.empty(max(hb, 1), dtype=torch.uint8, pin_memory=True)
    acc.event_begin, acc.event_end = ev[2].cuda_event, ev[3].cuda_event
    u = []
    for rep in range(reps + 2):
        flush()
        B.check(B.spec_accept(req, acc, (ws.data_ptr() + 255) // 256 * 256, db, stg.data_ptr(), hb,
                              torch.cuda.current_stream(dev).cuda_stream), "spec_accept")
        torch.cuda.synchronize()
        u.append(ev[2].elapsed_time(ev[3]) * 1e3)
    gem, tor = float(np.median(g[2:])), float(np.median(t[2:]))
    flops = 2.0 * M * K * V
    nbytes = V * K * 2 + M * K * 2 + M * V * (2 if pool.logit_dtype == W.BF16 else 4)
    out = {"rows": int(M), "hidden_dim": int(K), "vocab": int(V), "logits": pool.logit_dtype,
           "gemm_us": gem, "tflops": flops / gem / 1e6, "mfma_frac": flops / (gem * 1e-6) / MFMA_BF16_PEAK,
           "bytes": int(nbytes), "hbm_frac": nbytes / (gem * 1e-6) / 1e9 / HBM_PEAK_GBS,
           "torch_linear_bf16_us": tor,
           "accept_fused_us": float(np.median(a[2:])), "accept_unfused_us": float(np.median(u[2:]))}
    del lmv, b, ws
    torch.cuda.empty_cache()
    return out


HEADLINE = "ragged_gqa_b128"          # the largest workload that fits one GPU
OTHERS = ("mha7b_b32", "long_gqa_b8", "tree15_b64")


def measure_workload(name: str, seed: int, K: int, Wm: int, dev, flush, settle_s: float = 0.3) -> tuple:
    """Every GPU figure of one workload: warm and cold steps, the attention
    kernels alone (split + combine, packed and paged), the acceptance
    kernels alone (cold and warm; the row-statistics kernel alone; the
    sequential tree rule for trees).  Returns (figures, pool, outputs)."""
    import numpy as np
    import torch

    from paper_2505_17074_amd import binding as B
    from paper_2505_17074_amd import workload as W
    from paper_2505_17074_amd.batch import DeviceBatch, PagedKV, Verifier

    cfg = W.CONFIG_BY_NAME[name]
    print(f"[bench] {name}: drawing the seeded workload", file=sys.stderr, flush=True)
    pool = W.make_pool(cfg, seed)
    work = W.workload_bytes(pool)
    batch = DeviceBatch(pool, dev)
    ver = Verifier(batch)
    stream = torch.cuda.current_stream(dev)
    print(f"[bench] {name}: timing", file=sys.stderr, flush=True)

    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(K)]
    for e4 in ev:
        for e in e4:
            e.record(stream)          # materialise the events
    torch.cuda.synchronize()

    # Clocks settle first: the GPU's clocks ramp over the first tens of
    # milliseconds of work, so untimed steps run for `settle_s` of wall time
    # before the W warm-up steps (neither is timed; the timed region below is
    # exactly K steps).
    t_end = time.perf_counter() + settle_s
    while time.perf_counter() < t_end:
        for _ in range(20):
            ver.run("verify", stream)
        torch.cuda.synchronize()
    for _ in range(Wm):
        ver.run("verify", stream)
    torch.cuda.synchronize()

    # The timed region: K whole steps.  On every EVENT_EVERY-th step the
    # library records two events on the attention's launch stream, before the
    # split-KV kernel and after the split combine (the roofline's kernel
    # time); a marker on every step would itself cost the step several
    # microseconds.
    sampled = [k for k in range(K) if k % EVENT_EVERY == 0]
    t0 = time.perf_counter()
    for k in range(K):
        if k % EVENT_EVERY == 0:
            ver.attn.event_begin, ver.attn.event_end = ev[k][0].cuda_event, ev[k][1].cuda_event
        else:
            ver.attn.event_begin = ver.attn.event_end = None
        ver.run("verify", stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ver.attn.event_begin = ver.attn.event_end = None
    ms = (t1 - t0) * 1e3 / K
    attn_samples = [ev[k][0].elapsed_time(ev[k][1]) * 1e3 for k in sampled]
    t_attn_us = float(np.mean(attn_samples))

    # the attention kernels alone (spec_verify_attn, nothing beside them on
    # the GPU), next to the in-step figure above, where they share HBM with
    # the acceptance kernels on the side stream; events on the caller's
    # stream around each call give the whole call with its launch gaps
    for k in range(K):
        ver.attn.event_begin, ver.attn.event_end = ev[k][0].cuda_event, ev[k][1].cuda_event
        ev[k][2].record(stream)
        ver.run("attn", stream)
        ev[k][3].record(stream)
    torch.cuda.synchronize()
    ver.attn.event_begin = ver.attn.event_end = None
    alone = [ev[k][0].elapsed_time(ev[k][1]) * 1e3 for k in range(K)]
    t_alone_us = float(np.mean(alone))
    t_call_us = float(np.mean([ev[k][2].elapsed_time(ev[k][3]) for k in range(K)]) * 1e3)

    # The same attention alone and the same steps over a paged KV cache:
    # 64-token pages in a seeded random order, read through the block table.
    pk = PagedKV(batch, 64, seed=seed)
    pver = Verifier(batch, attn=pk.attn_args())
    for _ in range(Wm):
        pver.run("verify", stream)
    torch.cuda.synchronize()
    for k in range(K):
        pver.attn.event_begin, pver.attn.event_end = ev[k][0].cuda_event, ev[k][1].cuda_event
        pver.run("attn", stream)
    torch.cuda.synchronize()
    pver.attn.event_begin = pver.attn.event_end = None
    t_paged_us = float(np.mean([ev[k][0].elapsed_time(ev[k][1]) for k in range(K)]) * 1e3)
    t0 = time.perf_counter()
    for k in range(K):
        pver.run("verify", stream)
    torch.cuda.synchronize()
    ms_paged = (time.perf_counter() - t0) * 1e3 / K
    del pver, pk
    torch.cuda.empty_cache()

    # Cold steps: the same step after a flush of the caches, each timed by
    # events around the call on the caller's stream.  Back to back, every step
    # re-reads the same target logits, which the K/V stream (non-temporal
    # loads) leaves in the 256 MB Infinity Cache: the timed loop above is the
    # warm, steady state.
    KF = min(K, 50)
    for k in range(KF):
        flush()
        ev[k][0].record(stream)
        ver.run("verify", stream)
        ev[k][1].record(stream)
    torch.cuda.synchronize()
    cold = [ev[k][0].elapsed_time(ev[k][1]) * 1e3 for k in range(KF)]

    # the acceptance kernels alone (spec_accept), for their own roofline, each
    # call after a flush (cold) and, in a second loop, each after an untimed
    # attention call as in a step (warm: the logits stay cached)
    for _ in range(Wm):
        ver.run("accept", stream)
    torch.cuda.synchronize()
    for k in range(K):
        flush()
        ver.acc.event_begin, ver.acc.event_end = ev[k][2].cuda_event, ev[k][3].cuda_event
        ver.run("accept", stream)
    torch.cuda.synchronize()
    acc_cold = [ev[k][2].elapsed_time(ev[k][3]) * 1e3 for k in range(K)]
    t_acc_us = float(np.mean(acc_cold))
    for k in range(K):
        ver.run("attn", stream)
        ver.acc.event_begin, ver.acc.event_end = ev[k][2].cuda_event, ev[k][3].cuda_event
        ver.run("accept", stream)
    torch.cuda.synchronize()
    t_acc_warm_us = float(np.mean([ev[k][2].elapsed_time(ev[k][3]) for k in range(K)]) * 1e3)
    # token trees: the acceptance alone (cold) under sequential sibling verification
    t_acc_seq_us = None
    if pool.tree_parent is not None:
        ver.acc.tree_rule = B.SPEC_TREE_SEQUENTIAL
        for k in range(K):
            flush()
            ver.acc.event_begin, ver.acc.event_end = ev[k][2].cuda_event, ev[k][3].cuda_event
            ver.run("accept", stream)
        torch.cuda.synchronize()
        ver.acc.tree_rule = B.SPEC_TREE_INDEPENDENT
        ver.acc.event_begin = ver.acc.event_end = None
        t_acc_seq_us = float(np.mean([ev[k][2].elapsed_time(ev[k][3]) for k in range(K)]) * 1e3)
    # the row-statistics kernel alone (cold), in a loop of its own (an event
    # between the two acceptance kernels would lengthen the total above)
    for k in range(K):
        flush()
        ver.acc.event_begin, ver.acc.event_end, ver.acc.event_mid = ev[k][2].cuda_event, None, ev[k][4].cuda_event
        ver.run("accept", stream)
    torch.cuda.synchronize()
    ver.acc.event_begin = ver.acc.event_end = ver.acc.event_mid = None
    t_rows_us = float(np.mean([ev[k][2].elapsed_time(ev[k][4]) for k in range(K)]) * 1e3)
    # the acceptance's floor (spec_accept_floor_probe): the rows the row
    # statistics stream (under the shared-tree independent rule, the rows of
    # nodes with children), then the decision's chain of dependent round
    # trips, with none of the arithmetic; cold, like the acceptance above
    nreq = pool.batch
    floor_rows = int(pool.n_q.sum())
    if pool.tree_parent is not None and pool.tree_parents is None:
        inner = np.zeros(len(pool.tree_parent), bool)
        inner[np.asarray(pool.tree_parent)[1:]] = True
        floor_rows = nreq * int(inner.sum())
    eb = batch.logits.element_size()
    fws_bytes = B.spec_accept_floor_probe_bytes(pool.vocab, floor_rows, nreq)
    fws = torch.empty(fws_bytes, dtype=torch.uint8, device=dev)
    fout = torch.empty(nreq, dtype=torch.int32, device=dev)
    for k in range(K):
        flush()
        ev[k][2].record(stream)
        st = B.spec_accept_floor_probe(batch.logits.data_ptr(), batch.logits.stride(0), eb, pool.vocab, floor_rows,
                                       nreq, fws.data_ptr(), fws_bytes, fout.data_ptr(), stream.cuda_stream)
        B.check(st, "spec_accept_floor_probe")
        ev[k][3].record(stream)
    torch.cuda.synchronize()
    floor_cold = [ev[k][2].elapsed_time(ev[k][3]) * 1e3 for k in range(K)]
    t_floor_us = float(np.median(floor_cold))     # a few cold samples run far slower: the median
    del fws, fout

    # the outputs of the last (cold) step stand for every step: same inputs
    ver.run("verify", stream)
    res = ver.results()
    logit_bytes = int(work["Nq"]) * pool.vocab * (2 if pool.logit_dtype == W.BF16 else 4)
    achieved = work["attn_bytes"] / (t_attn_us * 1e-6) / 1e9
    # tokens a step emits: the accepted drafts plus the final token, per request
    emitted = int(res["accepted_len"].astype(np.int64).sum()) + pool.batch
    acc_read = W.accept_bytes_read(pool, res["accepted_node"])
    fig = {
        "value": work["Nq"] / (ms * 1e-3),
        "ms_per_step": ms,
        "config": {"workload": cfg.name, "requests": pool.batch, "verify_tokens": work["Nq"],
                   "kv_tokens": work["Nkv"], "q_heads": pool.num_q_heads, "kv_heads": pool.num_kv_heads,
                   "head_dim": pool.head_dim, "vocab": pool.vocab, "logits": pool.logit_dtype,
                   "tree_nodes": 0 if pool.tree_parent is None else len(pool.tree_parent), "seed": seed},
        "dtype": "bf16" if pool.qkv_dtype == W.BF16 else "f32",
        # the attention row of the path: the split-KV kernel and the split
        # combine, timed together by the library's events on their stream
        "roofline": {"bound": "hbm", "kernel": "attn_split_mfma + attn_combine", "achieved": achieved,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": measured_traffic(cfg.name),
                     "algorithmic_bytes": work["attn_bytes"], "kernel_us": t_attn_us,
                     "kernel_us_p10": pct(attn_samples, 10), "kernel_us_p90": pct(attn_samples, 90),
                     "kernel_us_alone": t_alone_us,
                     "kernel_us_alone_p10": pct(alone, 10), "kernel_us_alone_p90": pct(alone, 90),
                     "frac_alone": work["attn_bytes"] / (t_alone_us * 1e-6) / 1e9 / HBM_PEAK_GBS,
                     # the whole spec_verify_attn call alone, with its launch gaps
                     "call_us_alone": t_call_us,
                     "frac_call_alone": work["attn_bytes"] / (t_call_us * 1e-6) / 1e9 / HBM_PEAK_GBS,
                     # the same kernels over a paged KV cache (64-token pages, random order)
                     "paged": {"page_tokens": 64, "kernel_us_alone": t_paged_us,
                               "frac_alone": work["attn_bytes"] / (t_paged_us * 1e-6) / 1e9 / HBM_PEAK_GBS,
                               "ms_per_step": ms_paged},
                     "mfma_util": work["attn_flops"] / (t_attn_us * 1e-6) / MFMA_BF16_PEAK},
        "accepted_plus_bonus_tokens_per_s": emitted / (ms * 1e-3),
        "cold": {"steps": KF, "step_us_median": float(np.median(cold)), "step_us_p10": pct(cold, 10),
                 "step_us_p90": pct(cold, 90), "verified_tokens_per_s": work["Nq"] / (float(np.median(cold)) * 1e-6)},
        "accept": {"kernels_us": t_acc_us, "floor_us": t_floor_us, "floor_us_p10": pct(floor_cold, 10),
                   "floor_us_p90": pct(floor_cold, 90), "vs_floor": float(np.median(acc_cold)) / t_floor_us,
                   "kernels_us_p10": pct(acc_cold, 10),
                   "kernels_us_p90": pct(acc_cold, 90), "kernels_us_warm": t_acc_warm_us,
                   "kernels_us_sequential_tree": t_acc_seq_us,
                   "algorithmic_bytes_upper": work["accept_bytes"],
                   "achieved_GBs": work["accept_bytes"] / (t_acc_us * 1e-6) / 1e9,
                   "frac": work["accept_bytes"] / (t_acc_us * 1e-6) / 1e9 / HBM_PEAK_GBS,
                   # the rows this step's outcome needs (trees: the rows of nodes with
                   # children, and a chosen leaf's), priced the same way
                   "bytes_read": acc_read,
                   "frac_read": acc_read / (t_acc_us * 1e-6) / 1e9 / HBM_PEAK_GBS,
                   # the streaming kernel alone (every target logit once): begin -> mid event
                   "rowstats_us": t_rows_us, "rowstats_bytes": logit_bytes,
                   "rowstats_frac": logit_bytes / (t_rows_us * 1e-6) / 1e9 / HBM_PEAK_GBS},
    }
    del ver, batch
    torch.cuda.empty_cache()
    return fig, pool, res


def oracle_check(pool, res) -> dict:
    """The oracle against this step's GPU outputs (every request): accepted
    lengths, nodes and next tokens bit-exact except near ties (counted), and
    the attention's worst row-relative error over every output row, with the
    fraction of rows above 1e-3."""
    import numpy as np
    import oracle
    acc = oracle.verify_accept(pool.target_logits, pool.draft_probs, pool.draft_tokens, pool.uniforms, pool.n_q,
                               dtype=pool.logit_dtype, tree_parent=pool.tree_parent, tree_parents=pool.tree_parents)
    ties = acc["near_tie"]
    same = np.ones(pool.batch, bool)
    for key in ("accepted_len", "next_token", "accepted_node"):
        same &= np.asarray(res[key], np.int64) == acc[key]
    worst, rows, over = 0.0, 0, 0
    q0, kv0 = pool.q_start, pool.kv_start
    for i in range(pool.batch):
        n, c = int(pool.n_q[i]), int(pool.ctx_len[i])
        ref = oracle.verify_attention(pool.q[q0[i]:q0[i] + n], pool.k[kv0[i]:kv0[i + 1]], pool.v[kv0[i]:kv0[i + 1]],
                                      [c], [n], pool.num_kv_heads, dtype=pool.qkv_dtype,
                                      tree_parent=pool.parents_of(i))
        got = res["out"][q0[i]:q0[i] + n].astype(np.float64)
        r = np.abs(got - ref).max(-1) / np.abs(ref).max(-1)
        worst = max(worst, float(r.max()))
        rows += r.size
        over += int((r > 1e-3).sum())
    return {"requests": pool.batch, "near_ties": int(ties.sum()),
            "accept_mismatches_outside_ties": int((~same & ~ties).sum()),
            "accept_mismatches_at_ties": int((~same & ties).sum()),
            "attention_worst_row_rel_err": worst, "attention_rows": rows,
            "attention_frac_rows_over_1e-3": over / max(rows, 1), "attention_tolerance": 2e-3}


def main():
    args = parse()
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); multi-GPU sharding of the verify step is "
              "described in the design notes but not built", file=sys.stderr)
        sys.exit(2)
    import torch

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    flush = CacheFlush(dev)
    names = [args.workload] + ([] if args.only else [n for n in OTHERS + (HEADLINE,) if n != args.workload])
    figs, checks, head_pool = {}, {}, None
    for name in names:
        fig, pool, res = measure_workload(name, args.seed, args.steps, args.warmup, dev, flush, args.settle)
        figs[name] = fig
        if not args.no_cpu:
            # the cpu_baseline leg: the oracle's verdict on this step's outputs
            checks[name] = oracle_check(pool, res)
        if name == args.workload:
            head_pool = pool
        del pool, res
    if not args.no_lm_head:
        for name in names:
            figs[name]["lm_head"] = lm_head_figures(name, args.seed, dev, flush)
    del flush
    head = figs[args.workload]
    # the device's stream ceilings last: their 20 ms of full-rate reads and
    # copies leave the steps that follow them several percent slower
    read_ceiling, copy_rate = stream_ceilings_gbs(dev)
    for f in figs.values():
        f["roofline"]["stream_read_GBs"] = read_ceiling
        f["roofline"]["frac_of_stream_read"] = f["roofline"]["achieved"] / read_ceiling
        f["roofline"]["stream_copy_GBs"] = copy_rate

    line = {
        "metric": METRIC,
        "value": head["value"],
        "unit": "verified tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": head["dtype"],
        "data": "synthetic",
        "config": head["config"],
        "roofline": head["roofline"],
        "accepted_plus_bonus_tokens_per_s": head["accepted_plus_bonus_tokens_per_s"],
        "cache": "value and ms_per_step: back-to-back steps on the same inputs (warm: the target logits "
                 "stay in the Infinity Cache); cold: each step after a cache flush",
        "cold": head["cold"],
        "accept": head["accept"],
        "lm_head": head.get("lm_head"),
        # the other workloads, measured the same way in the same run
        "workloads": {n: f for n, f in figs.items() if n != args.workload},
    }
    if not args.no_sched:
        line["scheduler"] = scheduler_closed_loop(dev, args.seed)
    if not args.no_cpu:
        line["cpu_baseline"] = cpu_baseline(head_pool, args.cpu_seconds)
        line["cpu_baseline"]["oracle_check"] = checks
        if not args.no_sched:
            line["cpu_baseline"]["scheduler_oracle_decision_us"] = scheduler_oracle_decision_us(dev, args.seed)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
