"""CPU model of the exchange protocol of the sequential sibling kernel, run
before the kernel uses it.

C work-groups share one request's vocabulary.  At every exchange j (each
normaliser of a rejection, then the final sample's slice totals) a
work-group writes its value to slot (j, c), then adds one to the request's
counter, then waits until the counter reaches (j + 1) C and reads the C
slots of exchange j.  The counter starts at zero (the row-statistics kernel
clears it before the launch) and is never reset inside the call.

The model dispatches work-groups in launch order (request-major) into a
limited number of device slots, runs the dispatched ones in a random
interleaving, and checks, for every capacity of at least C slots:
  * every work-group finishes (no wait blocks forever);
  * at every exchange each work-group reads exactly the C values written for
    it, so all of a request's work-groups take the same decisions;
  * the counter ends at C x (exchanges), which the kernel's waits assume.
"""
import random

import pytest


def _worker(req, c, C, values, slots, counter, seen):
    """One work-group: yields while it waits; reads slots only after its wait."""
    for j, vals in enumerate(values):
        slots[req][(j, c)] = vals[c]          # write, then count the arrival
        yield
        counter[req] += 1
        yield
        while counter[req] < (j + 1) * C:     # the bounded spin on the device
            yield "wait"
        seen[(req, c, j)] = tuple(slots[req][(j, cc)] for cc in range(C))
        yield


def _run(n_req, C, exchanges, capacity, seed):
    rng = random.Random(seed)
    values = {r: [[rng.random() for _ in range(C)] for _ in range(exchanges[r])] for r in range(n_req)}
    slots = {r: {} for r in range(n_req)}
    counter = {r: 0 for r in range(n_req)}
    seen = {}
    order = [(r, c) for r in range(n_req) for c in range(C)]   # launch order
    pending = list(order)
    running = {}
    steps = 0
    while pending or running:
        while pending and len(running) < capacity:             # in-order dispatch
            r, c = pending.pop(0)
            running[(r, c)] = _worker(r, c, C, values[r], slots, counter, seen)
        key = rng.choice(list(running))
        steps += 1
        assert steps < 10_000_000, "no progress"
        try:
            next(running[key])
        except StopIteration:
            del running[key]
    return values, seen, counter


@pytest.mark.parametrize("C", [1, 2, 4, 8])
@pytest.mark.parametrize("seed", range(6))
def test_exchanges_complete_and_agree(C, seed):
    rng = random.Random(1000 + seed)
    n_req = rng.randint(1, 9)
    exchanges = [rng.randint(1, 6) for _ in range(n_req)]
    for capacity in sorted({C, C + 1, 2 * C + 1, C * n_req}):
        values, seen, counter = _run(n_req, C, exchanges, capacity, seed)
        for r in range(n_req):
            assert counter[r] == C * exchanges[r]
            for j in range(exchanges[r]):
                for c in range(C):
                    assert seen[(r, c, j)] == tuple(values[r][j])
