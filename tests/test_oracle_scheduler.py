"""Pins of the scheduler oracle against facts other than itself: the worked
example of Fig. 1, the optimality of shortest-job-first for simultaneous
arrivals (brute force over all orders), closed forms for least-attained-service
round robin and for the switching costs, hand-worked stability and Eq. (6)
values, the degenerate one-queue case, and the queue/no-preemption rules of
Sec. 4.2-4.3 on scenarios worked by hand."""
import itertools
import random

import pytest

from oracle.scheduler import Params, Request, eq6_estimate, queue_of, simulate


def _one_round(L, pred, us, arrival=0):
    # a request served in a single round that emits all L tokens
    return Request(arrival=arrival, prompt=0, out_len=L, pred_len=pred, draft=L - 1, round_us=us,
                   accepted=[L - 1] * L)


def test_fig1_worked_example():
    """Fig. 1 / Sec. 1: three requests arrive together; verification costs 10 ms
    per processed token (drafting omitted), so a request with output length L
    and acceptance rate A takes (L / A) x 10 ms.  R2 has L = 5 and A = 0.1:
    500 ms.  The printed averages (FCFS 583 ms, length-based SJF 683 ms,
    optimal 450 ms) fix the other two: FCFS gives 3 T1 + 2 T2 + T3 = 1750,
    the optimum (R3, R1, R2) 3 T3 + 2 T1 + T2 = 1350 and the length order
    (R2, R1, R3) 3 T2 + 2 T1 + T3 = 2050, whose solution is T1 = 200 ms and
    T3 = 150 ms.  Predicted lengths 10 and 12 for R1 and R3 (any
    5 < L1 < L3 gives the length order of the figure)."""
    reqs = [_one_round(10, 10, 200_000), _one_round(5, 5, 500_000), _one_round(12, 12, 150_000)]
    assert round(simulate(reqs, "fcfs")["avg_latency"] / 1000) == 583
    assert round(simulate(reqs, "lp_sjf")["avg_latency"] / 1000) == 683
    assert round(simulate(reqs, "sjf_exact")["avg_latency"] / 1000) == 450
    assert [e[0] for e in simulate(reqs, "lp_sjf")["log"]] == [1, 0, 2]
    assert [e[0] for e in simulate(reqs, "sjf_exact")["log"]] == [2, 0, 1]


@pytest.mark.parametrize("seed", range(20))
def test_sjf_exact_is_optimal_for_simultaneous_arrivals(seed):
    """Non-preemptive, all arriving at 0: shortest-first minimises the mean
    completion time (exchange argument) -- checked against every order."""
    rng = random.Random(seed)
    n = rng.randint(1, 6)
    reqs = []
    for _ in range(n):
        L = rng.randint(1, 6)
        reqs.append(Request(0, 0, L, rng.randint(1, 9), 2, rng.randint(1, 50),
                            [rng.randint(0, 2) for _ in range(L)]))
    got = simulate(reqs, "sjf_exact")["avg_latency"]
    times = []
    for r in reqs:                       # each request's total service, counted directly
        tok, k = 0, 0
        while tok < r.out_len:
            tok += r.accepted[k] + 1
            k += 1
        times.append(k * r.round_us)
    best = min(sum(itertools.accumulate(times[i] for i in order)) / n
               for order in itertools.permutations(range(n)))
    assert got == pytest.approx(best, abs=1e-9)
    assert simulate(reqs, "fcfs")["avg_latency"] >= best - 1e-9


@pytest.mark.parametrize("N,R,d", [(1, 3, 7), (3, 4, 10), (5, 2, 3)])
def test_las_identical_requests_round_robin(N, R, d):
    """Least attained service with identical requests arriving together and
    no switching cost: strict round robin, request i completes at
    (N (R - 1) + i + 1) d."""
    reqs = [Request(0, 0, R, R, 1, d, [0] * R) for _ in range(N)]
    out = simulate(reqs, "las")
    assert out["completion"] == [(N * (R - 1) + i + 1) * d for i in range(N)]
    assert [e[0] for e in out["log"]] == [i for _ in range(R) for i in range(N)]


def test_las_switching_costs_by_hand():
    """Two requests of two one-token rounds, prompt P, swap cost c per cached
    token each way: 0 runs, 1 preempts (0 swapped out with P + 1 tokens), 0
    resumes (1 out, 0 in), 0 finishes, 1 resumes (swapped in)."""
    P, c, d = 7, 3, 100
    reqs = [Request(0, P, 2, 2, 1, d, [0, 0]), Request(0, P, 2, 2, 1, d, [0, 0])]
    out = simulate(reqs, "las", Params(swap_us_per_token=c))
    s = c * (P + 1)
    assert out["completion"] == [3 * d + 3 * s, 4 * d + 4 * s]
    assert out["switches"] == 2 and out["switch_us"] == 4 * s
    assert [e[1] for e in out["log"]] == [0, d + s, 2 * d + 3 * s, 3 * d + 4 * s]


def test_eq6_closed_form():
    # n = 4, L = 100, A = 0.5, T_SSM = 2, T_LLM = 30: (800 + 3000) / 3
    assert eq6_estimate(4, 100, 0.5, 2, 30) == pytest.approx(3800 / 3, rel=1e-15)
    # A = 1 with one draft: every round yields 2 tokens -> L / 2 rounds
    assert eq6_estimate(1, 10, 1.0, 0, 8) == 40.0
    # no drafting: one token per round
    assert eq6_estimate(0, 10, 0.0, 5, 8) == 80.0


def test_queue_thresholds():
    p = Params(K=4, S1_up=100, M=2)        # [0,100) [100,200) [200,400) [400,inf)
    for E, j in [(0, 0), (99, 0), (100, 1), (199, 1), (200, 2), (399, 2), (400, 3), (10 ** 9, 3)]:
        assert queue_of(E, p) == j
    assert queue_of(10 ** 12, Params(K=1)) == 0


def test_stability_window_and_estimate_by_hand():
    """n = 4, accepted 4, 0, 2, 2, ...: running rates 1, 1/2, 1/2, 1/2, ...
    With gamma = 3 and delta = 0.01 the window [1/2, 1/2, 1/2] after round 4 is
    the first within delta: A = 1/2, T = (4*100*2 + 100*30) / 3."""
    r = Request(0, 0, 40, 100, 4, 10, [4, 0] + [2] * 38)
    p = Params(K=2, S1_up=10 ** 9, M=2, gamma=3, delta=0.01, t_ssm=2, t_llm=30)
    out = simulate([r], "laps_sd", p)
    assert out["perceptible"] == [True]
    assert out["A"] == [0.5]
    assert out["T_est"][0] == pytest.approx(3800 / 3, rel=1e-15)
    # never stable with gamma longer than the request, or delta = 0
    assert simulate([r], "laps_sd", Params(gamma=1000, delta=0.5))["perceptible"] == [False]
    assert simulate([r], "laps_sd", Params(gamma=2, delta=0.0))["perceptible"] == [False]


def _random_reqs(rng, n, max_arrival=2000):
    out = []
    for _ in range(n):
        L = rng.randint(1, 40)
        k = rng.randint(0, 6)
        out.append(Request(rng.randint(0, max_arrival), rng.randint(0, 50), L, rng.randint(1, 60), k,
                           rng.randint(5, 40), [rng.randint(0, k) for _ in range(L)]))
    return out


@pytest.mark.parametrize("seed", range(10))
def test_one_queue_without_stability_is_fcfs(seed):
    """K = 1 and delta = 0: one queue, nothing ever perceptible, so LAPS-SD
    serves non-perceptible requests first come first served, never
    preempting (the running request is always the earliest arrival)."""
    rng = random.Random(100 + seed)
    reqs = _random_reqs(rng, rng.randint(1, 12))
    p = Params(K=1, delta=0.0, swap_us_per_token=2)
    a, b = simulate(reqs, "laps_sd", p), simulate(reqs, "fcfs", p)
    assert a["log"] == b["log"] and a["completion"] == b["completion"] and a["switches"] == 0


def test_demotion_lets_a_new_request_in():
    """Queue 0 holds E < 25 us.  A (10 us rounds) reaches E = 30 after three
    rounds and drops to queue 1; B arrives at 25 into queue 0 and runs next,
    whether or not A has become perceptible (stable after two rounds)."""
    A = Request(0, 0, 30, 30, 4, 10, [2] * 30)          # 3 tokens per round: 10 rounds
    B = Request(25, 0, 1, 1, 0, 10, [0])
    for gamma in (1000, 2):
        out = simulate([A, B], "laps_sd", Params(K=2, S1_up=25, M=100, gamma=gamma, delta=0.01))
        assert out["perceptible"][0] == (gamma == 2)
        assert [e[0] for e in out["log"][:4]] == [0, 0, 0, 1] and out["completion"][1] == 40


def test_perceptible_not_preempted_inside_its_queue():
    """One effective queue: A becomes perceptible after two rounds and keeps
    the server when B arrives at 25, so B waits for A (110 us); least attained
    service hands the server to B at 30."""
    A = Request(0, 0, 30, 30, 4, 10, [2] * 30)
    B = Request(25, 0, 1, 1, 0, 10, [0])
    out = simulate([A, B], "laps_sd", Params(K=2, S1_up=10 ** 9, M=2, gamma=2, delta=0.01))
    assert [e[0] for e in out["log"]] == [0] * 10 + [1] and out["completion"] == [100, 110]
    assert [e[0] for e in simulate([A, B], "las")["log"][:4]] == [0, 0, 0, 1]


def test_perceptible_first_then_fcfs_by_hand():
    """Queue 0 holds E < 25 us; every request that drafts is stable after one
    round (gamma = 1).  F (never drafts, so never perceptible) runs 0-30 and
    drops to queue 1; G arrives at 1, runs 30-60 (perceptible after its first
    round) and drops too; H arrives at 55 into queue 0 and runs 60-70.  At 70
    queue 1 holds F (earlier arrival) and G: the perceptible G goes first
    (70-140), then F (140-210)."""
    F = Request(0, 0, 10, 10, 0, 10, [0] * 10)
    G = Request(1, 0, 20, 20, 4, 10, [1] * 20)
    H = Request(55, 0, 1, 1, 0, 10, [0])
    out = simulate([F, G, H], "laps_sd", Params(K=2, S1_up=25, M=100, gamma=1, delta=1.0))
    assert [e[0] for e in out["log"]] == [0, 0, 0, 1, 1, 1, 2] + [1] * 7 + [0] * 7
    assert out["completion"] == [210, 140, 70]
    assert out["perceptible"] == [False, True, False]


def test_sjf_among_perceptible_by_hand():
    """D1 (predicted 10 tokens) and D2 (predicted 1000) both draft 4 and accept
    1 per round (rate 1/4, stable after one round): Eq. (6) with T_SSM = 1,
    T_LLM = 10 gives 70 and 7000, both beyond queue 0's 25 us, so each moves
    to queue 1 as soon as it is perceptible.  D1 runs 0-10, D2 10-20 and then
    keeps the server (queue 1 is the top, and a running perceptible request
    is not preempted inside its queue) until E, arriving at 65 into queue 0,
    takes 70-80.  At 80 the shorter estimate, D1, goes first: its 29
    remaining rounds end at 370, then D2's 24 at 610."""
    D1 = Request(0, 0, 60, 10, 4, 10, [1] * 60)
    D2 = Request(0, 0, 60, 1000, 4, 10, [1] * 60)
    E = Request(65, 0, 1, 1, 0, 10, [0])
    out = simulate([D1, D2, E], "laps_sd", Params(K=2, S1_up=25, M=100, gamma=1, delta=1.0, t_ssm=1, t_llm=10))
    assert out["T_est"][:2] == [70.0, 7000.0]
    assert [e[0] for e in out["log"]] == [0] + [1] * 6 + [2] + [0] * 29 + [1] * 24
    assert out["completion"] == [370, 610, 80]


def test_estimate_places_a_perceptible_request():
    """Queue 0 holds service below 100 us, queue 1 below 400.  A drafts 4,
    accepts 2 per round (rate 1/2, stable after 2 rounds with gamma = 2):
    with T_LLM = 10 and predicted length 100, T = 100*10 / 3 = 333.3, so after
    its second round A sits in queue 1 although it has attained only 20 us,
    and B (arriving at 5, queue 0) runs next."""
    A = Request(0, 0, 30, 100, 4, 10, [2] * 30)
    B = Request(5, 0, 2, 2, 0, 10, [0, 0])
    out = simulate([A, B], "laps_sd", Params(K=3, S1_up=100, M=4, gamma=2, delta=0.01, t_llm=10))
    assert out["T_est"][0] == pytest.approx(1000 / 3, rel=1e-15)
    assert [e[0] for e in out["log"][:4]] == [0, 0, 1, 1]


@pytest.mark.parametrize("policy", ["fcfs", "lp_sjf", "sjf_exact", "las", "laps_sd"])
@pytest.mark.parametrize("seed", range(6))
def test_conservation(policy, seed):
    """Every request completes after its arrival; rounds never overlap and
    start no earlier than their request's arrival; the server is busy for
    exactly the rounds plus the switching; each request runs the number of
    rounds its trace needs."""
    rng = random.Random(seed)
    reqs = _random_reqs(rng, rng.randint(1, 15))
    p = Params(K=3, S1_up=60, M=3, gamma=3, delta=0.05, t_ssm=1, t_llm=20, swap_us_per_token=1)
    out = simulate(reqs, policy, p)
    log = out["log"]
    for (i, s, e), (_, s2, _) in zip(log, log[1:]):
        assert e <= s2
    busy = sum(e - s for _, s, e in log)
    for i, s, e in log:
        assert s >= reqs[i].arrival
    for i, r in enumerate(reqs):
        tok, k = 0, 0
        while tok < r.out_len:
            tok += min(r.accepted[k], r.draft) + 1
            k += 1
        assert sum(1 for j, _, _ in log if j == i) == k
        assert out["completion"][i] == max(e for j, _, e in log if j == i)
        assert out["latency"][i] >= k * r.round_us
    assert busy == sum(r.round_us * sum(1 for j, _, _ in log if j == i) for i, r in enumerate(reqs))
    # switching time is spent between rounds (never before the first)
    gaps = sum(s2 - e for (_, _, e), (_, s2, _) in zip(log, log[1:]))
    assert out["switch_us"] <= gaps


@pytest.mark.parametrize("policy", ["fcfs", "lp_sjf", "sjf_exact", "las", "laps_sd"])
def test_no_idle_gaps_without_switching_cost(policy):
    """All arriving at 0 and free switching: the server never idles."""
    rng = random.Random(7)
    reqs = _random_reqs(rng, 10, max_arrival=0)
    log = simulate(reqs, policy, Params(K=3, S1_up=60, M=3, gamma=3, delta=0.05))["log"]
    assert log[0][1] == 0 and all(e == s2 for (_, _, e), (_, s2, _) in zip(log, log[1:]))
