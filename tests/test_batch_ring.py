"""The Verifier's staging ring on the CPU: every rewrite of a staging slot
waits on an event recorded on the stream of that slot's last call, after that
call was issued, whatever mix of streams the caller uses.  Streams and events
are stand-ins that record the order of calls; no device is used."""
import random

import pytest

import paper_2505_17074_amd.batch as batch


class _Ev:
    last_on = {}                         # stream -> index of the last call issued on it
    records = 0

    def __init__(self):
        self.after = None
        self.stream = None

    def record(self, stream):
        _Ev.records += 1
        self.after = _Ev.last_on.get(stream)
        self.stream = stream

    def query(self):
        return True


class _FakeCuda:
    Event = _Ev


class _FakeTorch:
    cuda = _FakeCuda


class _Ring(batch.Verifier):
    def __init__(self, ring, every):      # the ring's state only: no workspace, no device
        self._staging = [None] * ring
        self._every = every
        self._slot_ev = [None] * ring
        self._pending = []
        self._pending_stream = None
        self._i = 0
        self._last_stream = None


@pytest.mark.parametrize("ring,every", [(32, 8), (8, 8), (9, 4), (4, 1), (64, 8)])
@pytest.mark.parametrize("streams", [("a",), ("a", "a", "a", "b", "c")])
def test_every_reuse_waits_on_a_covering_event(monkeypatch, ring, every, streams):
    monkeypatch.setattr(batch, "torch", _FakeTorch)
    _Ev.last_on = {}
    _Ev.records = 0
    rng = random.Random(ring * 31 + every)
    v = _Ring(ring, every)
    last = {}
    for i in range(3000):
        st = rng.choice(streams)
        s = v._slot(st)
        if s in last:
            j, sj = last[s]
            ev = v._slot_ev[s]
            assert ev is not None and ev.stream == sj and ev.after is not None and ev.after >= j, (i, s, j)
        _Ev.last_on[st] = i
        last[s] = (i, st)
        v._done(s, st)
    if len(streams) == 1:
        # one event per `every` calls on a single stream
        assert _Ev.records == v._i // every


def test_ring_shorter_than_event_period_is_refused():
    with pytest.raises(ValueError):
        batch.Verifier.__init__(object.__new__(batch.Verifier), None, ring=4, event_every=8)


class _Stream:
    """Stand-in stream: records the calls issued on it and the events it waits on."""

    def __init__(self, name):
        self.name = name
        self.waits = []

    def wait_event(self, ev):
        self.waits.append(ev)


def test_calls_on_another_stream_wait_for_the_previous_call(monkeypatch):
    """The workspace is shared by every call: a call on a stream other than
    the previous call's must be preceded, on its own stream, by a wait on an
    event recorded on the previous call's stream after that call."""
    monkeypatch.setattr(batch, "torch", _FakeTorch)
    _Ev.last_on = {}
    rng = random.Random(7)
    streams = [_Stream(n) for n in "abc"]
    v = _Ring(8, 4)
    prev = None
    for i in range(2000):
        st = rng.choice(streams)
        n_waits = len(st.waits)
        v._order(st)
        if prev is not None and st is not prev:
            assert len(st.waits) == n_waits + 1, i
            ev = st.waits[-1]
            assert ev.stream is prev and ev.after == _Ev.last_on[prev] == i - 1, i
        else:
            assert len(st.waits) == n_waits, i           # same stream: in order already
        _Ev.last_on[st] = i
        prev = st
