"""The host-side cooperative scheduler of local_sched.h (C++, in liblocal.so)
against its oracle (oracle/sched.py), call by call on seeded random operation
sequences; a discrete-event simulation of foreground requests arriving during
background chunks with safe boundaries (§4.2: foreground waits at most the
rest of the running non-yielding phase; nothing background starts while
foreground waits; every admitted chunk met §4.3's inequalities); and the error
behaviour of the C ABI. CPU only."""
import heapq

import numpy as np
import pytest

import paper_2608_15241_amd as lk
from oracle.sched import FOREGROUND, JUDGE, PREFILL, TRAIN, SchedOracle

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")

S = lk.Scheduler


def _random_task(rng):
    cls = int(rng.choice([FOREGROUND, JUDGE, TRAIN, PREFILL], p=[0.25, 0.25, 0.25, 0.25]))
    t = dict(cls=cls, priority=int(rng.integers(0, 3)), adapter=int(rng.integers(0, 4)),
             version=int(rng.integers(1, 5)),
             duration=float(rng.choice([-1.0, rng.uniform(0.001, 0.05)])),
             mem=float(rng.integers(0, 8)) * 1e9, max_nonyield=float(rng.uniform(0.0, 0.06)),
             utility=float(rng.integers(0, 4)), deadline=float(rng.choice(
                 [-1.0, rng.uniform(0.0, 2.0)])),
             tokens=int(rng.integers(1, 512)), prefix_len=int(rng.integers(0, 40000)))
    return t


@pytest.mark.parametrize("seed", range(6))
def test_random_sequences_match_the_oracle(seed):
    rng = np.random.default_rng(2000 + seed)
    params = dict(alpha_judge=float(rng.uniform(0.1, 1.0)), alpha_train=float(rng.uniform(0.1, 1)),
                  alpha_prefill=float(rng.uniform(0.1, 1.0)), reserve=float(rng.integers(0, 3)) * 1e9,
                  window=float(rng.uniform(0.02, 0.08)), delta=float(rng.uniform(0.0, 0.01)))
    s = S(params)
    o = SchedOracle(**params)
    now = 0.0
    for step in range(400):
        now += float(rng.uniform(0.0, 0.02))
        op = rng.choice(["submit", "submit", "next", "next", "finish", "cancel"])
        if op == "submit":
            t = _random_task(rng)
            i = s.submit(**t)
            assert i == o.submit(t)
            assert s.should_yield() == o.should_yield(), step
        elif op == "next":
            mem_free = float(rng.integers(0, 10)) * 1e9
            win = bool(rng.random() < 0.3)
            got = s.next(now, mem_free, win)
            want = o.next(now, mem_free, win)
            assert got[:2] == want[:2], (step, got, want)
            assert got[2] == pytest.approx(want[2], rel=1e-12, abs=0), step
            assert got[3] == pytest.approx(want[3], rel=1e-12, abs=0), step
        elif op == "finish":
            running = s.stats()[2]
            assert running == o.stats()[2]
            if running >= 0:
                if rng.random() < 0.7:
                    secs = float(rng.uniform(0.001, 0.05))
                    s.complete(running, secs)
                    o.complete(running, secs)
                else:
                    rq = bool(rng.random() < 0.7)
                    s.yield_(running, rq)
                    o.yield_(running, rq)
        elif op == "cancel":
            ids = [j for j, _ in o.queue]
            if ids:
                i = ids[int(rng.integers(len(ids)))]
                s.cancel(i)
                o.cancel(i)
        assert s.stats() == o.stats(), step
        L = int(rng.integers(0, 40000))
        for a, b in zip(s.estimates(L), o.estimates(L)):
            assert a == pytest.approx(b, rel=1e-12, abs=0), step


def test_simulated_foreground_waits_at_most_one_nonyielding_phase():
    """Training chunks made of non-yielding phases run between foreground
    requests; a foreground request arriving mid-phase is served as soon as
    that phase ends (the chunk stops at the boundary and is requeued)."""
    rng = np.random.default_rng(7)
    s = S(dict(window=0.060, delta=0.005, reserve=1e9))
    mem_free = 20e9
    events = []          # (time, order, kind, payload)
    order = 0
    for k in range(60):  # foreground arrivals
        t = float(rng.uniform(0.0, 3.0))
        events.append((t, order, "fg", None))
        order += 1
    heapq.heapify(events)
    chunk_phases = {}    # background chunk -> its remaining non-yielding phases
    chunk_meta = {}      # background chunk -> (memory, longest phase) as submitted
    for _ in range(20):  # background chunks queued up front
        phases = [float(rng.uniform(0.002, 0.04)) for _ in range(int(rng.integers(1, 6)))]
        mem = float(rng.integers(0, 6)) * 1e9
        i = s.submit(S.TRAIN, duration=sum(phases), mem=mem, max_nonyield=max(phases),
                     utility=float(rng.integers(0, 3)))
        chunk_phases[i] = phases
        chunk_meta[i] = (mem, max(phases))
    s.submit(S.TRAIN, duration=0.01, max_nonyield=0.08)   # never admissible: 80 + 5 > 60 ms
    now, running, phase_end, rest = 0.0, None, None, []
    fg_arrival, waits = {}, []
    fg_done = 0
    while fg_done < 60:
        # admit whatever may run now
        if running is None:
            d, tid, est, _ = s.next(now, mem_free)
            if d == S.RUN:
                if tid in fg_arrival:
                    waits.append(now - fg_arrival.pop(tid))
                    running, phase_end, rest = tid, now + 0.003, []
                else:
                    assert not fg_arrival, "background admitted while foreground waits"
                    mem, y = chunk_meta[tid]                  # §4.3 held at admission
                    assert mem + 1e9 <= mem_free and y + 0.005 <= 0.060
                    ph = chunk_phases[tid]
                    running, phase_end, rest = tid, now + ph[0], ph[1:]
        nxt_fg = events[0][0] if events else float("inf")
        if running is not None and phase_end <= nxt_fg:
            now = phase_end
            if running in chunk_phases and rest and not s.should_yield():
                chunk_phases[running] = rest
                phase_end, rest = now + rest[0], rest[1:]
                continue
            if running in chunk_phases and rest:         # safe boundary, yield requested
                chunk_phases[running] = rest
                s.yield_(running, True)
            else:
                s.complete(running, 0.01)
                if running not in chunk_phases:
                    fg_done += 1
            running = None
            continue
        if not events:
            break
        now, _, _, _ = heapq.heappop(events)
        fid = s.submit(S.FOREGROUND)
        fg_arrival[fid] = now
        if running is not None and running in chunk_phases:
            assert s.should_yield()
    assert fg_done == 60
    # one phase is at most 40 ms, a foreground task 3 ms: a request waits at
    # most the rest of one phase plus the foreground requests queued ahead
    assert max(waits) <= 0.040 + 0.003 * 60
    assert np.median(waits) <= 0.040


def test_errors_leave_the_scheduler_unchanged():
    with pytest.raises(lk.LocalError):
        S(dict(alpha_train=0.0))
    with pytest.raises(lk.LocalError):
        S(dict(window=-1.0))
    s = S()
    with pytest.raises(lk.LocalError):
        s.submit(7)                                    # no such class
    with pytest.raises(lk.LocalError):
        s.submit(S.JUDGE, mem=-1.0)
    with pytest.raises(lk.LocalError):
        s.submit(S.PREFILL, tokens=0)                  # nothing to estimate from
    with pytest.raises(lk.LocalError):
        s.complete(0, 0.1)                             # nothing running
    with pytest.raises(lk.LocalError):
        s.cancel(3)
    assert s.stats() == (0, 0, -1)
    i = s.submit(S.PREFILL, tokens=128, prefix_len=900, duration=-1.0)
    assert i == 0 and s.prefill_estimate(128, 900) == -1.0
    assert s.next(0.0, 1e9, True)[:2] == (S.RUN, 0)
    s.complete(0, 0.128)
    assert s.prefill_estimate(64, 1000) == pytest.approx(0.064)
    with pytest.raises(lk.LocalError):
        s.yield_(0)                                    # no longer running
