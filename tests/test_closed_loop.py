"""The closed loop: the verify step's accepted counts drive the native
scheduler.  CPU part: the workload recipe and a full evaluation on traces
drawn on the host.  GPU part: the traces come from the library's acceptance
kernels, whose first round is checked against the oracle."""
import numpy as np
import pytest

from paper_2505_17074_amd import closed_loop as CL


def _host_traces(cfg, wl, seed):
    rng = np.random.default_rng(seed)
    R = int(wl.out_len.max())
    level = rng.uniform(0.1, 0.9, size=cfg.requests)
    return rng.binomial(cfg.draft, level[:, None], size=(cfg.requests, R))


def test_workload_recipe():
    cfg = CL.LoopConfig(requests=40)
    wl = CL.make_workload(cfg, 0)
    assert (np.diff(wl.arrival) >= 0).all() and wl.arrival[0] >= 0
    assert (wl.out_len >= cfg.out_clip[0]).all() and (wl.out_len <= cfg.out_clip[1]).all()
    assert (wl.pred_len >= 1).all() and (wl.sigma >= cfg.sigma[0]).all() and (wl.sigma <= cfg.sigma[1]).all()
    again = CL.make_workload(cfg, 0)
    assert all(np.array_equal(getattr(wl, f), getattr(again, f)) for f in ("arrival", "out_len", "pred_len"))


def test_evaluate_on_host_traces():
    cfg = CL.LoopConfig(requests=30)
    wl = CL.make_workload(cfg, 1)
    reqs = CL.requests_from(cfg, wl, _host_traces(cfg, wl, 1))
    res = CL.evaluate(reqs, CL.default_params(cfg))
    assert set(res) == set(CL.POLICIES)
    for pol, r in res.items():
        assert r["avg_latency_ms"] > 0 and r["rounds"] >= len(reqs)
    assert res["fcfs"]["switches"] == 0 and res["lp_sjf"]["switches"] == 0
    assert res["laps_sd"]["perceptible"] > 0


@pytest.mark.gpu
def test_gpu_traces_match_the_oracle(gpu_lib):
    from oracle import verify_accept
    print("[case] closed-loop traces, 12 requests", flush=True)
    cfg = CL.LoopConfig(requests=12, vocab=512, out_median=40, out_clip=(4, 120))
    wl = CL.make_workload(cfg, 3)
    traces, first = CL.gpu_traces(cfg, wl, 3, capture_first=True)
    assert traces.shape[0] == cfg.requests and traces.min() >= 0 and traces.max() <= cfg.draft
    # every request emits its output length within the traced rounds
    assert ((traces + 1).sum(axis=1) >= wl.out_len).all()
    ref = verify_accept(first["target_logits"], first["draft_probs"], first["draft_tokens"], first["uniforms"],
                        [cfg.draft + 1] * cfg.requests)
    ok = ref["near_tie"] | ((ref["accepted_len"] == first["accepted_len"]) & (ref["next_token"] == first["next_token"]))
    assert ok.all()
    res = CL.evaluate(CL.requests_from(cfg, wl, traces), CL.default_params(cfg))
    assert all(r["avg_latency_ms"] > 0 for r in res.values())


def test_round_time_includes_the_measured_verify_kernels():
    """A request's round is n * T_SSM + T_LLM plus the verify kernels' time
    interpolated at its context (prompt plus half its output)."""
    cfg = CL.LoopConfig(requests=5, verify_us={128: 300.0, 2048: 1100.0})
    wl = CL.make_workload(cfg, 2)
    R = int(wl.out_len.max())
    reqs = CL.requests_from(cfg, wl, np.zeros((cfg.requests, R), np.int64))
    for i, r in enumerate(reqs):
        c = float(wl.prompt[i]) + wl.out_len[i] / 2
        extra = np.interp(c, [128, 2048], [300.0, 1100.0])
        assert r.round_us == cfg.draft * cfg.t_ssm_us + cfg.t_llm_us + int(round(extra))
    base = CL.requests_from(CL.LoopConfig(requests=5), wl, np.zeros((5, R), np.int64))
    assert all(b.round_us == cfg.draft * cfg.t_ssm_us + cfg.t_llm_us for b in base)


@pytest.mark.gpu
def test_measured_verify_times(gpu_lib):
    print("[case] closed-loop verify-kernel times", flush=True)
    t = CL.measure_verify("cuda", contexts=(128, 2048), reps=5)
    assert set(t) == {128, 2048} and all(np.isfinite(v) and v > 0 for v in t.values())
    assert t[2048] > t[128]            # 32 layers' attention over 16x the keys
