"""The library's native LAPS-SD scheduler (specsched.h) against the oracle:
every round of the schedule, every completion time, the switching totals and
the stability results must be identical -- integer times exactly, and the
acceptance rates and Eq. (6) estimates bit for bit, since both sides evaluate
them in the same order in fp64.  Host code only: these run without a GPU."""
import random

import pytest

from oracle.scheduler import Params, Request, simulate as oracle_simulate
from paper_2505_17074_amd import binding as B
from paper_2505_17074_amd.scheduler import SchedParams, SchedRequest, Scheduler, simulate

POLICIES = ["fcfs", "lp_sjf", "sjf_exact", "las", "laps_sd"]


def _workload(rng, n, max_arrival=3000, max_len=60, max_draft=8):
    reqs = []
    for _ in range(n):
        L = rng.randint(1, max_len)
        k = rng.randint(0, max_draft)
        # a per-request acceptance level, so that rates settle (or not)
        level = rng.random()
        acc = [sum(rng.random() < level for _ in range(k)) for _ in range(L)]
        reqs.append(Request(rng.randint(0, max_arrival), rng.randint(0, 300), L, rng.randint(1, 2 * max_len), k,
                            rng.randint(5, 60), acc))
    return reqs


def _params(rng):
    return Params(K=rng.randint(1, 6), S1_up=rng.randint(20, 500), M=rng.randint(2, 5), gamma=rng.randint(1, 6),
                  delta=rng.choice([0.0, 0.01, 0.05, 0.2, 1.0]), t_ssm=rng.randint(0, 3), t_llm=rng.randint(0, 50),
                  swap_us_per_token=rng.randint(0, 3))


def _native(reqs):
    return [SchedRequest(r.arrival, r.prompt, r.out_len, r.pred_len, r.draft, r.round_us, r.accepted) for r in reqs]


def _same(reqs, policy, p):
    ref = oracle_simulate(reqs, policy, p)
    got = simulate(_native(reqs), policy, p)
    assert got["log"] == ref["log"], policy
    for key in ("completion", "switches", "switch_us", "perceptible", "A", "T_est"):
        assert got[key] == ref[key], (policy, key)
    assert got["avg_latency"] == ref["avg_latency"]
    return ref


@pytest.mark.parametrize("policy", POLICIES)
@pytest.mark.parametrize("seed", range(40))
def test_random_workloads(policy, seed):
    rng = random.Random(1000 * seed + POLICIES.index(policy))
    _same(_workload(rng, rng.randint(1, 40)), policy, _params(rng))


@pytest.mark.parametrize("policy", POLICIES)
def test_edge_workloads(policy):
    rng = random.Random(5)
    one = _workload(rng, 1)
    together = _workload(rng, 12, max_arrival=0)
    twins = [Request(10, 5, 20, 20, 3, 17, [1] * 20) for _ in range(6)]          # all ties
    no_draft = _workload(rng, 10, max_draft=0)
    for reqs in (one, together, twins, no_draft):
        for p in (Params(), Params(K=1, gamma=1, delta=1.0), Params(K=6, S1_up=20, M=2, gamma=1, delta=0.0,
                                                                      swap_us_per_token=3, t_ssm=2, t_llm=40)):
            _same(reqs, policy, p)


@pytest.mark.parametrize("policy", POLICIES)
def test_large_workload(policy):
    rng = random.Random(77)
    reqs = _workload(rng, 300, max_arrival=200_000, max_len=120)
    ref = _same(reqs, policy, Params(K=5, S1_up=400, M=3, gamma=4, delta=0.03, t_ssm=2, t_llm=30,
                                     swap_us_per_token=1))
    assert sum(1 for _ in ref["log"]) > 1000


def test_online_api_matches_simulate():
    """A serving loop driving the online entry points (next / report) on the
    server model makes the same decisions as spec_sched_simulate."""
    rng = random.Random(9)
    reqs = _workload(rng, 25)
    p = SchedParams(K=4, S1_up=200, M=3, gamma=3, delta=0.05, t_ssm=1, t_llm=20, swap_us_per_token=0)
    ref = simulate(_native(reqs), "laps_sd", p)
    s = Scheduler("laps_sd", p, capacity=len(reqs))
    for r in reqs:
        s.submit(r.arrival, r.prompt, r.pred_len, r.draft)
    now, emitted, rounds, log = 0, [0] * len(reqs), [0] * len(reqs), []
    left = len(reqs)
    while left:
        i = s.next(now)
        if i < 0:
            now = min(r.arrival for j, r in enumerate(reqs) if emitted[j] < r.out_len)
            continue
        r = reqs[i]
        a = min(r.accepted[rounds[i]], r.draft)
        log.append((i, now, now + r.round_us))
        now += r.round_us
        rounds[i] += 1
        emitted[i] += a + 1
        fin = emitted[i] >= r.out_len
        left -= fin
        s.report(i, a, r.round_us, fin)
    assert log == ref["log"]
    for i in range(len(reqs)):
        q = s.query(i)
        assert q["finished"] and q["rounds"] == rounds[i]
        assert q["perceptible"] == ref["perceptible"][i] and q["T_est_us"] == ref["T_est"][i]
    s.close()


def test_argument_checks():
    lib = B.load()
    import ctypes as C
    h = C.c_void_p()
    good = SchedParams().to_c()
    for bad in (dict(K=0), dict(M=1), dict(S1_up=0), dict(gamma=0), dict(delta=-1.0), dict(delta=float("nan")),
                dict(t_llm=-1), dict(swap_us_per_token=-1)):
        p = SchedParams(**bad).to_c()
        assert lib.spec_sched_create(4, C.byref(p), 4, C.byref(h)) == B.SPEC_ERR_INVALID_ARG, bad
    assert lib.spec_sched_create(5, C.byref(good), 4, C.byref(h)) == B.SPEC_ERR_INVALID_ARG
    assert lib.spec_sched_create(0, C.byref(good), 0, C.byref(h)) == B.SPEC_ERR_INVALID_ARG
    s = Scheduler("las", SchedParams(), capacity=2)
    assert s.submit(0, 0, 5, 2) == 0 and s.submit(10, 0, 5, 2) == 1
    with pytest.raises(B.SpecError):
        s.submit(20, 0, 5, 2)                       # full
    with pytest.raises(B.SpecError):
        s.report(1, 0, 5, False)                    # not arrived yet
    assert s.next(0) == 0
    s.report(0, 1, 5, True)
    with pytest.raises(B.SpecError):
        s.report(0, 1, 5, False)                    # already finished
    assert s.next(5) == -1 and s.next(10) == 1
    bad = Scheduler("fcfs", SchedParams(), capacity=1)
    for args in ((-1, 0, 5, 2), (0, -1, 5, 2), (0, 0, 0, 2), (0, 0, 5, -1)):
        with pytest.raises(B.SpecError):
            bad.submit(*args)
    # a request whose trace is shorter than its output length, or a log too short
    r = SchedRequest(0, 0, 5, 5, 2, 10, [1, 1])
    with pytest.raises(B.SpecError):
        simulate([r], "fcfs")
