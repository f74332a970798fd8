"""CPU model of the attention kernel's item-claim protocol, run under random
interleavings of its atomic steps.

The claim word holds (call tag << 32) | next item.  Work-group 0 installs
(tag << 32) | first_round by compare-and-swap unless the word already holds
the tag; every later work-group takes one fetch-and-add, and on meeting
another tag polls the word a bounded number of times for the install, then
falls back to a compare-and-swap loop that starts the count itself; the
work-group that draws the grid's last index resets the word to
(tag << 32) | first_round so that a replay of the same launch (same tag)
claims from the first round again.  Each step below is one atomic operation
on the word; a schedule interleaves the work-groups' steps at random.

Checked for every schedule: the claims are exactly first_round .. grid - 1,
each once; every work-group finishes; the word ends as (tag << 32) |
first_round, ready for a replay; and a replay and a call with a new tag
behave the same.  (The protocol's steps are restated here from its
description; no code is shared with the kernel.)
"""
import random

import pytest

MASK64 = (1 << 64) - 1
MASK32 = (1 << 32) - 1


def _start_wg0(tag, base):
    """Work-group 0: load, then compare-and-swap while the tag differs."""
    old = yield ("load",)
    while (old >> 32) != tag:
        ok, old = yield ("cas", old, (tag << 32) | base)
        if ok:
            return None
    return None


def _claimer(tag, base, grid, polls, out):
    old = yield ("add",)
    if (old >> 32) == tag:
        idx = old & MASK32
    else:
        idx = None
        for _ in range(polls):
            old = yield ("load",)
            if (old >> 32) == tag:
                old = yield ("add",)
                idx = old & MASK32
                break
        if idx is None:
            old = yield ("load",)
            while True:
                nw = old + 1 if (old >> 32) == tag else (tag << 32) | (base + 1)
                ok, old2 = yield ("cas", old, nw & MASK64)
                if ok:
                    idx = (nw & MASK32) - 1
                    break
                old = old2
    if idx == grid - 1:
        yield ("store", (tag << 32) | base)
    out.append(idx)
    return None


def _run(word, tag, base, grid, polls, rng, wg0_delay=0):
    """One launch: work-group 0 (which also takes item 0 statically) and the
    claimers base .. grid - 1, interleaved at random.  Returns (claims, word)."""
    claims = []
    agents = [_start_wg0(tag, base)] + [_claimer(tag, base, grid, polls, claims) for _ in range(base, grid)]
    pending = {i: None for i in range(len(agents))}     # the value to send into each agent
    started = set()
    live = list(range(len(agents)))
    steps = 0
    while live:
        steps += 1
        assert steps < 100000, "a schedule did not finish"
        choices = [i for i in live if i != 0 or steps > wg0_delay] or live
        i = rng.choice(choices)
        g = agents[i]
        try:
            op = g.send(pending[i]) if i in started else next(g)
            started.add(i)
        except StopIteration:
            live.remove(i)
            continue
        kind = op[0]
        if kind == "load":
            pending[i] = word
        elif kind == "add":
            pending[i] = word
            word = (word + 1) & MASK64
        elif kind == "cas":
            _, expect, new = op
            if word == expect:
                pending[i] = (True, word)
                word = new
            else:
                pending[i] = (False, word)
        elif kind == "store":
            word = op[1]
            pending[i] = None
    return claims, word


@pytest.mark.parametrize("seed", range(40))
def test_claims_are_each_item_once_in_any_interleaving(seed):
    rng = random.Random(seed)
    base = rng.choice([1, 2, 5, 16])
    grid = base + rng.randint(1, 40)
    polls = rng.choice([0, 1, 3, 64])
    tag = rng.randint(1, MASK32)
    # the word's previous contents: junk, the previous call's final state, or
    # junk that only differs from this call's tag
    word = rng.choice([rng.getrandbits(64), ((tag - 1) & MASK32) << 32 | base,
                       ((tag ^ 1) << 32) | rng.getrandbits(32)])
    wg0_delay = rng.choice([0, 5, 50, 10000])           # work-group 0 late, even after every claim
    claims, word = _run(word, tag, base, grid, polls, rng, wg0_delay)
    assert sorted(claims) == list(range(base, grid)), (seed, sorted(claims))
    assert word == (tag << 32) | base
    # a replay of the same launch (same tag, the word as the call left it)
    claims, word = _run(word, tag, base, grid, polls, rng, wg0_delay)
    assert sorted(claims) == list(range(base, grid))
    assert word == (tag << 32) | base
    # the next call, with a new tag
    tag2 = (tag + 1) & MASK32 or 1
    claims, word = _run(word, tag2, base, grid, polls, rng)
    assert sorted(claims) == list(range(base, grid))
    assert word == (tag2 << 32) | base


def test_a_replay_without_the_reset_would_skip_items():
    """The reset matters: a word left at the end of its count with the same
    tag hands out indices past the grid on the next launch (the model of the
    protocol without the last claimer's store)."""
    tag, base, grid = 7, 2, 10
    word = (tag << 32) | grid                             # where the count ends
    rng = random.Random(0)
    claims = []
    g = _claimer(tag, base, grid, 0, claims)
    op = next(g)
    assert op == ("add",)
    try:
        g.send(word)
    except StopIteration:
        pass
    assert claims == [grid]                               # past the last item: nothing claimed


def _arrival(tag, total, lasts):
    """One piece of a split stream checks in: load, then compare-and-swap
    (old + 1 under the call's tag, else (tag << 32) | 1); the piece that
    makes the count `total` is the stream's last and resets the counter to
    (tag << 32) | 0 for a replay with the same tag."""
    old = yield ("load",)
    while True:
        nw = old + 1 if (old >> 32) == tag else (tag << 32) | 1
        ok, old2 = yield ("cas", old, nw & MASK64)
        if ok:
            break
        old = old2
    if (nw & MASK32) == total:
        yield ("store", tag << 32)
        lasts.append(1)
    return None


def _run_arrivals(word, tag, total, rng):
    lasts = []
    agents = [_arrival(tag, total, lasts) for _ in range(total)]
    pending = {i: None for i in range(total)}
    started, live = set(), list(range(total))
    while live:
        i = rng.choice(live)
        try:
            op = agents[i].send(pending[i]) if i in started else next(agents[i])
            started.add(i)
        except StopIteration:
            live.remove(i)
            continue
        if op[0] == "load":
            pending[i] = word
        elif op[0] == "cas":
            if word == op[1]:
                pending[i] = (True, word)
                word = op[2]
            else:
                pending[i] = (False, word)
        else:
            word = op[1]
    return len(lasts), word


@pytest.mark.parametrize("seed", range(30))
def test_split_stream_has_exactly_one_last_piece(seed):
    """The split combine's arrival counter: whatever the interleaving and the
    counter's previous contents, exactly one piece is the stream's last, on
    the call, on a replay with the same tag, and on the next call."""
    rng = random.Random(1000 + seed)
    total = rng.randint(1, 48)
    tag = rng.randint(1, MASK32)
    word = rng.choice([rng.getrandbits(64), ((tag - 1) & MASK32) << 32 | total, tag << 32])
    for t in (tag, tag, (tag + 1) & MASK32 or 1):
        n_last, word = _run_arrivals(word, t, total, rng)
        assert n_last == 1, (seed, t)
        assert word == t << 32
