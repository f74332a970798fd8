"""Closed-loop evaluation of the scheduler on the verify step's own accepted
counts (the LAPS-SD setting of Sec. 3 and Sec. 5: requests served one at a
time in speculative decoding rounds).

Each request drafts n tokens per round.  For every round index r, the drafts
of all requests are verified in ONE batched call of the library's acceptance
kernels (spec_accept): target and draft logits are synthetic and seeded, the
target row being the draft row plus N(0, sigma_i^2) noise, so request i has
an acceptance level of its own (sigma_i small: high acceptance).  The
accepted counts of rounds 0, 1, ... form each request's trace; the trace of
a request does not depend on when it is served, so one pass over the rounds
serves every policy.  The native scheduler (specsched.h) then serves the
workload under each policy on the server model of Sec. 3.

Times (integer microseconds):
  * a round lasts n * T_SSM + T_LLM + t_verify(c): T_LLM = 10 ms per
    verification (the per-token verification time Fig. 1 assumes for
    LLaMA-7B) stands for the target forward outside the verify kernels,
    T_SSM = 0.5 ms per drafted token, and t_verify(c) is MEASURED on the GPU
    by `measure_verify`: the verify attention of each of LLaMA-7B's 32
    decoder layers plus one acceptance, for one request whose context is c
    (the request's prompt plus half its output);
  * switching swaps a request's KV cache at `swap_us_per_token` per cached
    token each way.  The default of 8 us assumes LLaMA-7B fp16 KV (512 KB
    per token) over a 64 GB/s host link; `measure_swap` times the copies on
    the machine at hand, and the benchmark uses its figure.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional

import numpy as np

from . import binding as B
from .scheduler import SchedParams, SchedRequest, simulate

POLICIES = ("fcfs", "lp_sjf", "las", "laps_sd", "sjf_exact")


@dataclasses.dataclass
class LoopConfig:
    requests: int = 50                 # the paper varies 10..50 (Sec. 5.2)
    draft: int = 4                     # n
    vocab: int = 1024
    draft_logit_std: float = 2.0
    sigma: tuple = (0.3, 3.0)          # per-request target-noise range (uniform)
    out_median: int = 200              # true output length: log-normal, median, sigma, clip
    out_sigma: float = 0.8
    out_clip: tuple = (8, 1500)
    pred_sigma: float = 0.5            # predictor error: pred = out * exp(N(0, pred_sigma^2))
    prompt: tuple = (32, 512)
    t_ssm_us: int = 500
    t_llm_us: int = 10_000
    swap_us_per_token: int = 8
    arrival_frac: float = 0.3          # arrivals uniform over this fraction of the total service
    layers: int = 32                   # LLaMA-7B decoder layers: one verify attention each per round
    verify_us: Optional[dict] = None   # measured {context: us} of one round's verify kernels (None: not counted)


@dataclasses.dataclass
class LoopWorkload:
    arrival: np.ndarray
    prompt: np.ndarray
    out_len: np.ndarray
    pred_len: np.ndarray
    sigma: np.ndarray


KV_BYTES_PER_TOKEN = 2 * 32 * 4096 * 2     # LLaMA-7B: K and V, 32 layers, 4096 wide, fp16


def measure_swap(device="cuda", tokens=(16, 64, 256, 1024, 4096), reps: int = 5) -> dict:
    """KV swap cost on this machine (the switching cost of Sec. 3, Fig. 3):
    device -> pinned host and host -> device copies of a request's KV cache
    (KV_BYTES_PER_TOKEN per token), timed by events on the current stream.
    Returns GB/s per direction and size, and the cost per cached token at the
    largest size (both directions averaged), rounded up to whole us."""
    import torch
    top = max(tokens) * KV_BYTES_PER_TOKEN
    dev = torch.empty(top, dtype=torch.uint8, device=device)
    host = torch.empty(top, dtype=torch.uint8, pin_memory=True)
    dev.fill_(1)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    out = {"d2h_GBs": {}, "h2d_GBs": {}}
    for t in tokens:
        nb = t * KV_BYTES_PER_TOKEN
        for name, dst, src in (("d2h_GBs", host, dev), ("h2d_GBs", dev, host)):
            dst[:nb].copy_(src[:nb], non_blocking=True)
            e0.record()
            for _ in range(reps):
                dst[:nb].copy_(src[:nb], non_blocking=True)
            e1.record()
            torch.cuda.synchronize()
            out[name][t] = nb * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    t = max(tokens)
    gbs = 2.0 / (1.0 / out["d2h_GBs"][t] + 1.0 / out["h2d_GBs"][t])
    out["us_per_token"] = int(np.ceil(KV_BYTES_PER_TOKEN / (gbs * 1e9) * 1e6))
    del dev, host
    return out


def measure_verify(device="cuda", contexts=(128, 512, 1024, 2048), reps: int = 20, layers: int = 32,
                   draft: int = 4) -> dict:
    """One round's verify kernels on this GPU, per context length: the
    library's verify attention for each of `layers` decoder layers plus one
    acceptance, for one request of the LLaMA-7B shape (32 heads x 128,
    `draft` drafts, vocabulary 32000, bf16 KV cache, fp32 logits), timed by
    events around spec_verify_attn and spec_accept calls.  Returns
    {context: us}."""
    import dataclasses as dc
    import torch
    from . import workload as W
    from .batch import DeviceBatch, Verifier
    base = W.CONFIG_BY_NAME["mha7b_b32"]
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    out = {}
    for c in contexts:
        cfg = dc.replace(base, name=f"verify_c{c}", batch=1, ctx=("const", int(c)), draft=("const", draft))
        b = DeviceBatch(W.make_pool(cfg, 0), device)
        v = Verifier(b)
        t = {}
        for which in ("attn", "accept"):
            for _ in range(3):
                v.run(which)
            e0.record()
            for _ in range(reps):
                v.run(which)
            e1.record()
            torch.cuda.synchronize()
            t[which] = e0.elapsed_time(e1) * 1e3 / reps
        out[int(c)] = layers * t["attn"] + t["accept"]
        del v, b
    return out


def verify_us_at(cfg: LoopConfig, context: float) -> int:
    """t_verify at a context length, interpolated in the measured table (0 when none)."""
    if not cfg.verify_us:
        return 0
    xs = sorted(cfg.verify_us)
    return int(round(float(np.interp(context, xs, [cfg.verify_us[x] for x in xs]))))


def make_workload(cfg: LoopConfig, seed: int) -> LoopWorkload:
    rng = np.random.default_rng(np.random.SeedSequence([2505_17074, seed]))
    n = cfg.requests
    out = np.clip(np.rint(cfg.out_median * np.exp(cfg.out_sigma * rng.standard_normal(n))), *cfg.out_clip)
    pred = np.maximum(1, np.rint(out * np.exp(cfg.pred_sigma * rng.standard_normal(n))))
    sigma = rng.uniform(*cfg.sigma, size=n)
    prompt = rng.integers(cfg.prompt[0], cfg.prompt[1] + 1, size=n)
    # arrivals spread over a fraction of the expected total service (about
    # 2.5 tokens per round), so that requests queue
    round_us = cfg.draft * cfg.t_ssm_us + cfg.t_llm_us
    total = float(np.sum(out / 2.5 * round_us))
    arrival = np.sort(rng.uniform(0.0, cfg.arrival_frac * total, size=n)).astype(np.int64)
    return LoopWorkload(arrival, prompt.astype(np.int64), out.astype(np.int64), pred.astype(np.int64), sigma)


def gpu_traces(cfg: LoopConfig, wl: LoopWorkload, seed: int, device="cuda", capture_first: bool = False):
    """Accepted counts [requests, rounds] from the library's acceptance
    kernels, one batched spec_accept call per round index, until every
    request has emitted its output length.  With capture_first, also the
    first round's inputs and outputs (host copies), for checking."""
    import torch
    n, k, V = cfg.requests, cfg.draft, cfg.vocab
    g = torch.Generator(device=device)
    g.manual_seed(int(2505_17074 + seed))
    req = B.make_requests(np.zeros(n, np.int32), np.full(n, k, np.int32))
    Nq = n * (k + 1)
    logits = torch.empty((Nq, V), dtype=torch.float32, device=device)
    probs = torch.empty((n * k, V), dtype=torch.float32, device=device)
    tokens = torch.empty(n * k, dtype=torch.int32, device=device)
    uniforms = torch.empty(Nq, dtype=torch.float32, device=device)
    acc_len = torch.empty(n, dtype=torch.int32, device=device)
    nxt = torch.empty(n, dtype=torch.int32, device=device)
    a = B.SpecAcceptArgs()
    a.vocab, a.dtype = V, B.SPEC_F32
    a.target_logits, a.logits_stride = logits.data_ptr(), V
    a.draft_probs, a.probs_stride = probs.data_ptr(), V
    a.draft_tokens, a.uniforms = tokens.data_ptr(), uniforms.data_ptr()
    a.accepted_len, a.next_token = acc_len.data_ptr(), nxt.data_ptr()
    st, dev_bytes, host_bytes = B.spec_workspace_bytes(req, None, a)
    B.check(st, "spec_workspace_bytes")
    ws = torch.empty(dev_bytes + 256, dtype=torch.uint8, device=device)
    ws_ptr = (ws.data_ptr() + 255) // 256 * 256
    staging = torch.empty(max(host_bytes, 1), dtype=torch.uint8, pin_memory=True)
    sig = torch.tensor(np.repeat(wl.sigma, k + 1), dtype=torch.float32, device=device)[:, None]
    stream = torch.cuda.current_stream(device)
    emitted = np.zeros(n, np.int64)
    rows = []
    first = None
    while (emitted < wl.out_len).any():
        d = torch.randn((Nq, V), generator=g, device=device) * cfg.draft_logit_std
        logits.copy_(d + sig * torch.randn((Nq, V), generator=g, device=device))
        q = torch.softmax(d.view(n, k + 1, V)[:, :k], dim=-1).reshape(n * k, V)
        probs.copy_(q)
        tokens.copy_(torch.multinomial(q, 1, generator=g).view(-1).to(torch.int32))
        uniforms.copy_(torch.rand(Nq, generator=g, device=device))
        B.check(B.spec_accept(req, a, ws_ptr, dev_bytes, staging.data_ptr(), host_bytes, stream.cuda_stream),
                "spec_accept")
        torch.cuda.synchronize(device)          # the staging buffer is reused next round
        r = acc_len.cpu().numpy().astype(np.int64)
        if capture_first and first is None:
            first = {"target_logits": logits.cpu().numpy(), "draft_probs": probs.cpu().numpy(),
                     "draft_tokens": tokens.cpu().numpy(), "uniforms": uniforms.cpu().numpy(),
                     "accepted_len": r.copy(), "next_token": nxt.cpu().numpy()}
        rows.append(r)
        emitted += r + 1
    traces = np.stack(rows, axis=1)
    return (traces, first) if capture_first else traces


def requests_from(cfg: LoopConfig, wl: LoopWorkload, traces: np.ndarray) -> List[SchedRequest]:
    out = []
    for i in range(cfg.requests):
        L = int(wl.out_len[i])
        acc = np.zeros(max(L, traces.shape[1]), np.int64)
        acc[:traces.shape[1]] = traces[i]
        round_us = cfg.draft * cfg.t_ssm_us + cfg.t_llm_us + verify_us_at(cfg, int(wl.prompt[i]) + L / 2)
        out.append(SchedRequest(int(wl.arrival[i]), int(wl.prompt[i]), L, int(wl.pred_len[i]), cfg.draft, round_us,
                                acc))
    return out


def default_params(cfg: LoopConfig, K: int = 3) -> SchedParams:
    """K = 3 queues from 800 ms of service up by a factor 2; the acceptance
    rate is stable once 3 rounds differ by less than 0.05.  (The paper gives
    no values; these were the best of a sweep over K, S1_up, M, gamma and
    delta on workload seeds 10-15 of this recipe, host-drawn traces.)"""
    return SchedParams(K=K, S1_up=800_000, M=2, gamma=3, delta=0.05, t_ssm=cfg.t_ssm_us, t_llm=cfg.t_llm_us,
                       swap_us_per_token=cfg.swap_us_per_token)


def evaluate(reqs: List[SchedRequest], params: SchedParams) -> dict:
    """Mean latency (ms) and switching totals of every policy."""
    res = {}
    for pol in POLICIES:
        o = simulate(reqs, pol, params, log=False)
        res[pol] = {"avg_latency_ms": o["avg_latency"] / 1000.0, "switches": o["switches"],
                    "switch_ms": o["switch_us"] / 1000.0, "rounds": o["n_rounds"],
                    "perceptible": int(sum(o["perceptible"]))}
    return res
