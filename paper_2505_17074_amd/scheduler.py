"""Python face of the library's LAPS-SD scheduler (specsched.h): argument
marshalling only, every decision is made by the native scheduler.

`Scheduler` is the online form a serving loop drives (submit requests, ask
for the request of the next round, report the round's accepted count);
`simulate` serves a whole workload of accepted-count traces on the paper's
one-request-at-a-time server model and returns completion times and the
round log.
"""
from __future__ import annotations

import ctypes as C
import dataclasses
from typing import Sequence

import numpy as np

from . import binding as B


@dataclasses.dataclass
class SchedParams:
    K: int = 4                   # priority queues
    S1_up: int = 100_000         # us: upper threshold of the first queue
    M: int = 4                   # threshold ratio between consecutive queues
    gamma: int = 5               # rounds in the stability window
    delta: float = 0.02          # stability threshold on max - min of the window
    t_ssm: int = 0               # us per drafted token (Eq. (6))
    t_llm: int = 0               # us per verification pass (Eq. (6))
    swap_us_per_token: int = 0   # KV swap cost per cached token, each direction

    def to_c(self) -> B.SpecSchedParams:
        c = B.SpecSchedParams()
        c.K, c.M, c.S1_up_us, c.gamma = self.K, self.M, self.S1_up, self.gamma
        c.delta, c.t_ssm_us, c.t_llm_us = float(self.delta), self.t_ssm, self.t_llm
        c.swap_us_per_token = self.swap_us_per_token
        return c


@dataclasses.dataclass
class SchedRequest:
    arrival: int                 # us
    prompt: int                  # tokens in the KV cache at arrival
    out_len: int                 # true output length
    pred_len: int                # predicted output length
    draft: int                   # drafted tokens per round
    round_us: int                # duration of each of its rounds
    accepted: Sequence[int]      # accepted count of each round (>= out_len entries)


def _params(p) -> B.SpecSchedParams:
    if isinstance(p, SchedParams):
        return p.to_c()
    return SchedParams(p.K, p.S1_up, p.M, p.gamma, p.delta, p.t_ssm, p.t_llm, p.swap_us_per_token).to_c()


class Scheduler:
    """One native scheduler object (not thread-safe)."""

    def __init__(self, policy: str, params=None, capacity: int = 1024):
        self._params = _params(params or SchedParams())
        h = C.c_void_p()
        B.check(B.load().spec_sched_create(B.SCHED_POLICY[policy], C.byref(self._params), capacity, C.byref(h)),
                "spec_sched_create")
        self._h = h

    def close(self):
        if self._h:
            B.load().spec_sched_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def submit(self, arrival: int, prompt: int, pred_len: int, draft: int, size_hint: int = 0) -> int:
        i = C.c_int32(-1)
        B.check(B.load().spec_sched_submit(self._h, arrival, prompt, pred_len, draft, size_hint, C.byref(i)),
                "spec_sched_submit")
        return i.value

    def next(self, now: int) -> int:
        i = C.c_int32(-1)
        B.check(B.load().spec_sched_next(self._h, now, C.byref(i)), "spec_sched_next")
        return i.value

    def report(self, rid: int, accepted: int, round_us: int, finished: bool) -> None:
        B.check(B.load().spec_sched_report(self._h, rid, int(accepted), int(round_us), 1 if finished else 0),
                "spec_sched_report")

    def query(self, rid: int) -> dict:
        st = B.SpecSchedState()
        B.check(B.load().spec_sched_query(self._h, rid, C.byref(st)), "spec_sched_query")
        return {"attained_us": st.attained_us, "queue": st.queue, "perceptible": bool(st.perceptible),
                "finished": bool(st.finished), "rounds": st.rounds, "A": st.A, "T_est_us": st.T_est_us}


def simulate(reqs, policy: str, params=None, log: bool = True) -> dict:
    """Serve `reqs` (objects with the SchedRequest fields) to completion with
    the native scheduler; the same result layout as a round-by-round model."""
    n = len(reqs)
    arr = (B.SpecSchedRequest * n)()
    keep = []
    max_rounds = 0
    for i, r in enumerate(reqs):
        acc = np.ascontiguousarray(r.accepted, dtype=np.int32)
        keep.append(acc)
        q = arr[i]
        q.arrival_us, q.round_us, q.prompt_tokens = r.arrival, r.round_us, r.prompt
        q.out_len, q.pred_len, q.draft = r.out_len, r.pred_len, r.draft
        q.accepted = acc.ctypes.data_as(C.POINTER(C.c_int32))
        q.n_accepted = int(acc.shape[0])
        max_rounds += int(r.out_len)            # at least one token per round
    completion = np.zeros(n, np.int64)
    perc = np.zeros(n, np.int32)
    A = np.zeros(n, np.float64)
    T = np.zeros(n, np.float64)
    res = B.SpecSchedResult()
    res.completion_us = completion.ctypes.data_as(C.POINTER(C.c_int64))
    if log:
        rreq = np.zeros(max_rounds, np.int32)
        rstart = np.zeros(max_rounds, np.int64)
        res.round_req = rreq.ctypes.data_as(C.POINTER(C.c_int32))
        res.round_start_us = rstart.ctypes.data_as(C.POINTER(C.c_int64))
        res.max_rounds = max_rounds
    res.perceptible = perc.ctypes.data_as(C.POINTER(C.c_int32))
    res.A = A.ctypes.data_as(C.POINTER(C.c_double))
    res.T_est_us = T.ctypes.data_as(C.POINTER(C.c_double))
    P = _params(params or SchedParams())
    B.check(B.load().spec_sched_simulate(arr, n, B.SCHED_POLICY[policy], C.byref(P), C.byref(res)),
            "spec_sched_simulate")
    nr = int(res.n_rounds)
    out = {"completion": [int(x) for x in completion],
           "latency": [int(completion[i]) - int(reqs[i].arrival) for i in range(n)],
           "switches": int(res.switches), "switch_us": int(res.switch_us), "n_rounds": nr,
           "perceptible": [bool(x) for x in perc], "A": [float(x) for x in A], "T_est": [float(x) for x in T]}
    out["avg_latency"] = sum(out["latency"]) / n
    if log:
        out["log"] = [(int(rreq[k]), int(rstart[k]), int(rstart[k]) + int(reqs[int(rreq[k])].round_us))
                      for k in range(nr)]
    return out
