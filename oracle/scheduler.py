"""Plain round-by-round simulator of the LAPS-SD request scheduler and its
baselines (test infrastructure).

TEST INFRASTRUCTURE ONLY: imported by the test suite and the benchmark's
CPU-baseline leg, never by the product path, and sharing no code with the
library's native scheduler.

The serving model (Sec. 3: one request served at a time, "batch size 1").
  * Request i arrives at r_i with a prompt of P_i tokens; it must emit Lt_i
    tokens (its true output length), and the scheduler knows only a predicted
    length Lp_i (the output of the length predictor of Sec. 4.3, an input
    here).  It drafts n_i tokens per round.
  * One speculative decoding round of request i (Sec. 2.2): the SSM drafts
    n_i tokens and the LLM verifies them in one pass.  The round lasts
    `round_us[i]` (n_i * T_SSM + T_LLM for the workloads here) and emits
    a + 1 tokens, where a = the round's accepted count (the verify step's
    output) and the +1 is the LLM's additional token (Sec. 4.3).  The request
    completes at the end of the round in which its emitted total reaches Lt_i.
  * Switching (Sec. 3, Fig. 3): when the server moves from an unfinished
    request to another, the preempted request's KV cache is swapped out, and
    a request resumed after a preemption has its KV cache swapped in.  Each
    transfer costs `swap_us_per_token` x (P + tokens emitted so far) and
    occupies the server.  A request's attained service E_i counts only its
    rounds, i.e. speculation plus verification (Sec. 4.2).
  * All times are integers (microseconds), so completion times are exact.

Policies (`policy`):
  "fcfs"       non-preemptive, earliest arrival first (Sec. 1, Fig. 1(a)).
  "lp_sjf"     non-preemptive, smallest predicted output length first
               (Sec. 5.1 baseline, Fig. 1(b)).
  "sjf_exact"  non-preemptive, smallest true execution time first (the
               optimum of Fig. 1(c) for simultaneous arrivals).
  "las"        least attained service first, re-decided after every round
               (Sec. 3, Sec. 5.1 baseline).
  "laps_sd"    Algorithm 1 (Sec. 4.1-4.3):
      - K queues; queue j (0-based here) covers service times S with
        S_down(j) <= S < S_up(j), where S_up(j) = S1_up * M^j for j < K-1,
        the last queue is unbounded, S_down(j) = S_up(j-1) and
        S_down(0) = 0.  New requests enter queue 0.  After every round a
        non-perceptible request moves to the queue holding its attained
        service E (Sec. 4.2); a perceptible one to the queue holding
        max(E, T), its Eq. (6) estimate T ("moved to the corresponding
        queue", Sec. 4.1), so that attained service takes over only if it
        overruns its estimate.
      - The highest non-empty queue is served (inter-queue, Sec. 4.2).
      - Within it, perceptible requests go first, shortest estimated
        execution time first (SJF); then non-perceptible ones, earliest
        arrival first (FCFS) (intra-queue, Sec. 4.3).
      - A running perceptible request keeps the server while its queue is
        the highest non-empty one (SJF without preemption inside a queue);
        every other choice is re-made after every round, so a request in a
        higher queue, or the running request's own demotion, still ends its
        turn.
      - Stability (Sec. 4.3): after each round the running acceptance rate
        (accepted drafts so far / drafted tokens so far) is recorded; once the
        last gamma recorded rates differ by less than delta (max - min), the
        request becomes perceptible with A = the mean of those gamma rates and
        the execution time estimate of Eq. (6):
            T = (n * Lp * T_SSM + Lp * T_LLM) / (n * A + 1).

Readings of points the paper leaves open:
  * M is an integer >= 2, so every threshold is an exact integer.
  * A perceptible request is placed by max(E, T) (above): its estimate
    puts it in the queue it is expected to finish in, which is why, in the
    paper's words, perceptible requests seldom exceed their queue's
    threshold.  "No preemption" holds inside a queue only: were a
    perceptible request never preempted at all, it would run to completion
    from the round it became perceptible, and the SJF order among
    perceptible requests could never act.
  * The SJF key is the Eq. (6) estimate itself (the paper's "request size"),
    not a remaining-time estimate; ties go to the earlier arrival, then the
    smaller index.
  * The acceptance-rate denominator is the drafted tokens (the +1 token is not
    a draft); a request that drafts nothing (n = 0) never becomes perceptible.
  * Every other tie goes to the earlier arrival, then the smaller index.

Floating point appears only in the rates, the stability test and Eq. (6).
The operations and their order are fixed by the formulas above:
  * rate = accepted / drafted;
  * A = (left-to-right sum of the window) / gamma;
  * T = float(n*Lp*T_SSM + Lp*T_LLM) / (float(n) * A + 1.0);
  * the queue of a perceptible request uses T truncated to an integer.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence

POLICIES = ("fcfs", "lp_sjf", "sjf_exact", "las", "laps_sd")


@dataclasses.dataclass
class Request:
    arrival: int                 # us
    prompt: int                  # tokens already in the KV cache at arrival
    out_len: int                 # true output length Lt (tokens to emit), >= 1
    pred_len: int                # predicted output length Lp, >= 1
    draft: int                   # n: drafted tokens per round, >= 0
    round_us: int                # duration of one of its rounds, >= 1
    accepted: Sequence[int]      # accepted count of each round (clamped to [0, n])


@dataclasses.dataclass
class Params:
    K: int = 4                   # priority queues
    S1_up: int = 100_000         # us: upper threshold of the first queue
    M: int = 4                   # threshold ratio between consecutive queues
    gamma: int = 5               # rounds in the stability window
    delta: float = 0.02          # stability threshold on max - min of the window
    t_ssm: int = 0               # us per drafted token (Eq. (6))
    t_llm: int = 0               # us per verification pass (Eq. (6))
    swap_us_per_token: int = 0   # KV swap cost per cached token, each direction


def eq6_estimate(n: int, pred_len: int, A: float, t_ssm: int, t_llm: int) -> float:
    """Eq. (6): speculation time n*L*T_SSM plus verification time L*T_LLM, over
    the n*A + 1 tokens a round is expected to yield."""
    return float(n * pred_len * t_ssm + pred_len * t_llm) / (float(n) * A + 1.0)


def queue_of(E: int, p: Params) -> int:
    """Index of the queue whose [S_down, S_up) range holds attained service E."""
    up = p.S1_up
    for j in range(p.K - 1):
        if E < up:
            return j
        up *= p.M
    return p.K - 1


def simulate(reqs: List[Request], policy: str, p: Optional[Params] = None) -> dict:
    """Serve every request; returns completion times, the round log and
    switching totals."""
    if policy not in POLICIES:
        raise ValueError(policy)
    p = p or Params()
    N = len(reqs)
    for r in reqs:
        if r.out_len < 1 or r.round_us < 1 or r.draft < 0 or len(r.accepted) < r.out_len:
            raise ValueError("request needs out_len >= 1, round_us >= 1 and >= out_len accepted counts")
    done = [False] * N
    emitted = [0] * N
    rounds = [0] * N
    E = [0] * N                        # attained service (rounds only)
    swapped = [False] * N              # KV cache swapped out after a preemption
    acc_sum = [0] * N
    drafted = [0] * N
    rates: List[List[float]] = [[] for _ in range(N)]
    perceptible = [False] * N
    A = [0.0] * N
    T_est = [0.0] * N
    queue = [0] * N
    total_exec = [None] * N
    if policy == "sjf_exact":
        for i, r in enumerate(reqs):       # rounds needed with the true trace
            tok, k = 0, 0
            while tok < r.out_len:
                tok += min(max(int(r.accepted[k]), 0), r.draft) + 1
                k += 1
            total_exec[i] = k * r.round_us
    completion = [0] * N
    log = []                            # (request, round start, round end)
    n_switch, switch_us = 0, 0
    now = 0
    running: Optional[int] = None       # the request whose KV is resident

    def pick(ready: List[int]) -> int:
        if policy in ("fcfs", "lp_sjf", "sjf_exact") and running is not None and not done[running]:
            return running
        if policy == "fcfs":
            return min(ready, key=lambda i: (reqs[i].arrival, i))
        if policy == "lp_sjf":
            return min(ready, key=lambda i: (reqs[i].pred_len, reqs[i].arrival, i))
        if policy == "sjf_exact":
            return min(ready, key=lambda i: (total_exec[i], reqs[i].arrival, i))
        if policy == "las":
            return min(ready, key=lambda i: (E[i], reqs[i].arrival, i))
        # laps_sd
        top = min(queue[i] for i in ready)
        if running is not None and not done[running] and perceptible[running] and queue[running] == top:
            return running
        cand = [i for i in ready if queue[i] == top]
        perc = [i for i in cand if perceptible[i]]
        if perc:
            return min(perc, key=lambda i: (T_est[i], reqs[i].arrival, i))
        return min(cand, key=lambda i: (reqs[i].arrival, i))

    while not all(done):
        ready = [i for i in range(N) if not done[i] and reqs[i].arrival <= now]
        if not ready:
            now = min(reqs[i].arrival for i in range(N) if not done[i])
            continue
        i = pick(ready)
        if running is not None and running != i and not done[running]:
            cost = p.swap_us_per_token * (reqs[running].prompt + emitted[running])
            swapped[running] = True
            now += cost
            switch_us += cost
            n_switch += 1
        if swapped[i]:
            cost = p.swap_us_per_token * (reqs[i].prompt + emitted[i])
            swapped[i] = False
            now += cost
            switch_us += cost
        r = reqs[i]
        a = min(max(int(r.accepted[rounds[i]]), 0), r.draft)
        start = now
        now += r.round_us
        log.append((i, start, now))
        rounds[i] += 1
        emitted[i] += a + 1
        E[i] += r.round_us
        running = i
        if emitted[i] >= r.out_len:
            done[i] = True
            completion[i] = now
            continue
        if policy == "laps_sd":
            if not perceptible[i] and r.draft > 0:
                acc_sum[i] += a
                drafted[i] += r.draft
                rates[i].append(acc_sum[i] / drafted[i])
                if len(rates[i]) >= p.gamma:
                    win = rates[i][-p.gamma:]
                    if max(win) - min(win) < p.delta:
                        perceptible[i] = True
                        s = 0.0
                        for x in win:
                            s += x
                        A[i] = s / p.gamma
                        T_est[i] = eq6_estimate(r.draft, r.pred_len, A[i], p.t_ssm, p.t_llm)
            queue[i] = queue_of(max(E[i], int(T_est[i])) if perceptible[i] else E[i], p)
    latency = [completion[i] - reqs[i].arrival for i in range(N)]
    return {"completion": completion, "latency": latency,
            "avg_latency": sum(latency) / N if N else 0.0,
            "log": log, "switches": n_switch, "switch_us": switch_us,
            "perceptible": perceptible, "A": A, "T_est": T_est}
