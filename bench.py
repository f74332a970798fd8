"""Benchmark of the batched speculative-decoding verify step on one MI355X.

A step is one spec_verify call over one batch: host plan (staged), split-KV
verify attention (+ combine), acceptance and the final sample -- every row of
the hot path -- over inputs already resident in HBM.  Prints ONE JSON line.

  python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu]
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
    ap.add_argument("--workload", default="mha7b_b32")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-sched", action="store_true",
                    help="skip the scheduler's closed loop (thousands of small launches; for profiler runs)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
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
    cfg = CL.LoopConfig(swap_us_per_token=swap["us_per_token"])
    wl = CL.make_workload(cfg, seed)
    t0 = time.perf_counter()
    traces = CL.gpu_traces(cfg, wl, seed, device=dev)
    t_traces = time.perf_counter() - t0
    reqs = CL.requests_from(cfg, wl, traces)
    params = CL.default_params(cfg)
    res = CL.evaluate(reqs, params)
    lat = {pol: r["avg_latency_ms"] for pol, r in res.items()}
    sweep = {K: simulate(reqs, "laps_sd", CL.default_params(cfg, K=K), log=False)["avg_latency"] / 1000.0
             for K in (1, 2, 3, 4, 6, 8, 10)}
    reps, t0 = 20, time.perf_counter()
    for _ in range(reps):
        o = simulate(reqs, "laps_sd", params, log=False)
    dec_us = (time.perf_counter() - t0) / reps / o["n_rounds"] * 1e6
    return {"workload": f"{cfg.requests} requests, draft {cfg.draft}, output lengths log-normal (median "
                        f"{cfg.out_median}), predicted with log-normal error sigma {cfg.pred_sigma}, per-request "
                        f"acceptance from target noise sigma in {list(cfg.sigma)}; rounds "
                        f"{cfg.draft} x {cfg.t_ssm_us} + {cfg.t_llm_us} us; KV swap {cfg.swap_us_per_token} us/token",
            "rounds_traced": int(traces.shape[1]), "trace_s": t_traces,
            "mean_tokens_per_round": float((traces + 1).mean()),
            "avg_latency_ms": lat,
            "laps_sd_vs": {pol: lat[pol] / lat["laps_sd"] for pol in ("fcfs", "lp_sjf", "las", "sjf_exact")},
            "switches": {pol: r["switches"] for pol, r in res.items()},
            "laps_sd_perceptible": res["laps_sd"]["perceptible"],
            "laps_sd_avg_latency_ms_by_K": sweep,
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


def kernel_source_digest() -> str:
    h = hashlib.sha256()
    for name in ("attention.hip", "sv_internal.h"):
        with open(os.path.join(ROOT, "paper_2505_17074_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload: str):
    """HBM bytes per launch of the split-KV kernel from the committed rocprofv3
    counter summary, if it was taken on the current kernel source."""
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
                                [c], [n], pool.num_kv_heads, dtype=pool.qkv_dtype, tree_parent=pool.tree_parent)
        oracle.verify_accept(pool.target_logits[q0[i]:q0[i] + n], pool.draft_probs[pool.d_start[i]:pool.d_start[i + 1]],
                             pool.draft_tokens[q0[i] - i:q0[i] - i + n - 1], pool.uniforms[q0[i]:q0[i] + n], [n],
                             dtype=pool.logit_dtype, tree_parent=pool.tree_parent)
        t_used += time.perf_counter() - t0
        done_tokens += n
        m += 1
    return {"value": done_tokens / t_used, "unit": "verified tokens/s", "cores": int(threads), "cpu_model": cpu_model(),
            "kind": "oracle",
            "sample": f"{m} request verifications ({m / pool.batch:.2f} passes over the {pool.batch} requests, "
                      f"{done_tokens} verify tokens), attention + acceptance in fp64 NumPy, {t_used:.1f} s"}


def main():
    args = parse()
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); multi-GPU sharding of the verify step is "
              "described in the design notes but not built", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2505_17074_amd import binding as B
    from paper_2505_17074_amd import workload as W
    from paper_2505_17074_amd.batch import DeviceBatch, Verifier

    cfg = W.CONFIG_BY_NAME[args.workload]
    pool = W.make_pool(cfg, args.seed)
    work = W.workload_bytes(pool)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    batch = DeviceBatch(pool, dev)
    ver = Verifier(batch)
    stream = torch.cuda.current_stream(dev)

    K, Wm = args.steps, args.warmup
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(K)]
    for e4 in ev:
        for e in e4:
            e.record(stream)          # materialise the events
    torch.cuda.synchronize()

    for _ in range(Wm):
        ver.run("verify", stream)
    torch.cuda.synchronize()

    # The timed region: K whole steps.  On every EVENT_EVERY-th step the
    # library records two events immediately around the split-KV attention
    # kernel on its launch stream (the roofline's kernel time); a marker on
    # every step would itself cost the step several microseconds.
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

    # the attention kernel alone (spec_verify_attn, nothing beside it on the
    # GPU), for its own roofline next to the in-step figure above, where it
    # shares HBM with the acceptance kernels on the side stream; events on the
    # caller's stream around each call give the whole call (split
    # kernel, split combine)
    for k in range(K):
        ver.attn.event_begin, ver.attn.event_end = ev[k][0].cuda_event, ev[k][1].cuda_event
        ev[k][2].record(stream)
        ver.run("attn", stream)
        ev[k][3].record(stream)
    torch.cuda.synchronize()
    ver.attn.event_begin = ver.attn.event_end = None
    t_alone_us = float(np.mean([ev[k][0].elapsed_time(ev[k][1]) for k in range(K)]) * 1e3)
    t_call_us = float(np.mean([ev[k][2].elapsed_time(ev[k][3]) for k in range(K)]) * 1e3)

    # The same attention alone and the same steps over a paged KV cache:
    # 64-token pages in a seeded random order, read through the block table.
    from paper_2505_17074_amd.batch import PagedKV
    pk = PagedKV(batch, 64, seed=args.seed)
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
    flush = CacheFlush(dev)
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
    t_acc_us = float(np.mean([ev[k][2].elapsed_time(ev[k][3]) for k in range(K)]) * 1e3)
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
    del flush
    logit_bytes = int(work["Nq"]) * pool.vocab * (2 if pool.logit_dtype == W.BF16 else 4)
    achieved = work["attn_bytes"] / (t_attn_us * 1e-6) / 1e9
    traffic = measured_traffic(args.workload)
    # tokens a step emits: the accepted drafts plus the final token, per request
    # (the same inputs every step, so the last step's outputs stand for all)
    emitted = int(batch.accepted_len.to(torch.int64).sum().item()) + pool.batch
    acc_read = W.accept_bytes_read(pool, batch.accepted_node.cpu().numpy())
    # the device's stream ceilings last: their 20 ms of full-rate reads and
    # copies leave the steps that follow them several percent slower
    read_ceiling, copy_rate = stream_ceilings_gbs(dev)

    line = {
        "metric": METRIC,
        "value": work["Nq"] / (ms * 1e-3),
        "unit": "verified tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": Wm,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if pool.qkv_dtype == W.BF16 else "f32",
        "data": "synthetic",
        "config": {"workload": cfg.name, "requests": pool.batch, "verify_tokens": work["Nq"],
                   "kv_tokens": work["Nkv"], "q_heads": pool.num_q_heads, "kv_heads": pool.num_kv_heads,
                   "head_dim": pool.head_dim, "vocab": pool.vocab, "logits": pool.logit_dtype,
                   "tree_nodes": 0 if pool.tree_parent is None else len(pool.tree_parent), "seed": args.seed},
        "roofline": {"bound": "hbm", "kernel": "attn_split_mfma", "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "algorithmic_bytes": work["attn_bytes"], "kernel_us": t_attn_us,
                     "kernel_us_p10": pct(attn_samples, 10), "kernel_us_p90": pct(attn_samples, 90),
                     "kernel_us_alone": t_alone_us,
                     "frac_alone": work["attn_bytes"] / (t_alone_us * 1e-6) / 1e9 / HBM_PEAK_GBS,
                     # the whole spec_verify_attn call alone: split + combine, with their launch gaps
                     "call_us_alone": t_call_us,
                     # the same kernel over a paged KV cache (64-token pages, random order)
                     "paged": {"page_tokens": 64, "kernel_us_alone": t_paged_us,
                               "frac_alone": work["attn_bytes"] / (t_paged_us * 1e-6) / 1e9 / HBM_PEAK_GBS,
                               "ms_per_step": ms_paged},
                     "frac_call_alone": work["attn_bytes"] / (t_call_us * 1e-6) / 1e9 / HBM_PEAK_GBS,
                     "mfma_util": work["attn_flops"] / (t_attn_us * 1e-6) / MFMA_BF16_PEAK,
                     "stream_read_GBs": read_ceiling, "frac_of_stream_read": achieved / read_ceiling,
                     "stream_copy_GBs": copy_rate},
        "accepted_plus_bonus_tokens_per_s": emitted / (ms * 1e-3),
        "cache": "value and ms_per_step: back-to-back steps on the same inputs (warm: the target logits "
                 "stay in the Infinity Cache); cold: each step after a cache flush",
        "cold": {"steps": KF, "step_us_median": float(np.median(cold)), "step_us_p10": pct(cold, 10),
                 "step_us_p90": pct(cold, 90), "verified_tokens_per_s": work["Nq"] / (float(np.median(cold)) * 1e-6)},
        "accept": {"kernels_us": t_acc_us, "kernels_us_warm": t_acc_warm_us,
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
    if not args.no_sched:
        line["scheduler"] = scheduler_closed_loop(dev, args.seed)
    if not args.no_cpu:
        line["cpu_baseline"] = cpu_baseline(pool, args.cpu_seconds)
        if not args.no_sched:
            line["cpu_baseline"]["scheduler_oracle_decision_us"] = scheduler_oracle_decision_us(dev, args.seed)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
