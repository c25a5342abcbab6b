"""Pins of the scheduler oracle (§4) against closed forms and hand-worked cases:
the moving average's geometric weights, the prefix-length buckets at their
edges, the admissibility inequalities on both sides of each bound, foreground
priority and the yield request, the no-sample rule, and the offload decision."""
import pytest

from oracle.sched import (BUCKETS, FOREGROUND, IDLE, JUDGE, OFFLOAD, PREFILL, RUN, TRAIN,
                          BUSY, SchedOracle, bucket)


def task(cls, **kw):
    t = dict(cls=cls, priority=0, adapter=0, version=0, duration=-1.0, mem=0.0,
             max_nonyield=0.0, utility=0.0, deadline=-1.0, tokens=0, prefix_len=0)
    t.update(kw)
    return t


def run_and_complete(o, t, seconds, now=0.0):
    i = o.submit(t)
    d, j, _, _ = o.next(now, 1e12, True)
    assert (d, j) == (RUN, i)
    o.complete(i, seconds)


def test_moving_average_has_geometric_weights():
    # E_k = (1-a)^(k-1) v_1 + sum_{i>=2} a (1-a)^(k-i) v_i
    a = 0.25
    vs = [0.8, 0.2, 0.5, 1.1, 0.05]
    o = SchedOracle(alpha_train=a)
    for v in vs:
        run_and_complete(o, task(TRAIN), v)
    k = len(vs)
    closed = (1 - a) ** (k - 1) * vs[0] + sum(a * (1 - a) ** (k - i) * vs[i - 1]
                                              for i in range(2, k + 1))
    assert o.estimates(0)[1] == pytest.approx(closed, rel=1e-14)
    # a constant series stays constant; alpha = 1 keeps the last sample
    o = SchedOracle(alpha_judge=1.0)
    for v in (3.0, 7.0):
        run_and_complete(o, task(JUDGE), v)
    assert o.estimates(0)[0] == 7.0


def test_prefill_buckets_and_rate():
    assert [bucket(L) for L in (0, 1, 512, 513, 1024, 1025, 32768, 32769, 10 ** 6)] == \
        [0, 0, 0, 1, 1, 2, 6, 6, 6]
    assert BUCKETS[-1] == 32768
    o = SchedOracle(alpha_prefill=0.5)
    run_and_complete(o, task(PREFILL, tokens=128, prefix_len=700), 0.064)  # 0.5 ms/token
    run_and_complete(o, task(PREFILL, tokens=256, prefix_len=1000), 0.256)  # 1 ms/token
    assert o.estimates(1024)[2] == pytest.approx(0.75e-3)                  # same bucket
    assert o.estimates(512)[2] == -1.0 and o.estimates(2048)[2] == -1.0    # others unset
    assert o.estimate(task(PREFILL, tokens=64, prefix_len=600)) == pytest.approx(0.048)


def test_admissibility_bounds():
    # reserve 1 GB, window 50 ms, margin 5 ms
    o = SchedOracle(reserve=1e9, window=0.050, delta=0.005)
    i = o.submit(task(JUDGE, duration=0.010, mem=2e9, max_nonyield=0.045))
    assert o.next(0.0, 3e9, False)[:2] == (RUN, i)              # 2 + 1 <= 3, 45 + 5 <= 50
    o.complete(i, 0.010)
    i = o.submit(task(JUDGE, duration=0.010, mem=2e9, max_nonyield=0.0451))
    assert o.next(0.0, 1e12, False)[0] == IDLE                  # 45.1 + 5 > 50
    o.cancel(i)
    i = o.submit(task(JUDGE, duration=0.010, mem=2e9 + 1, max_nonyield=0.0))
    d, j, _, deficit = o.next(0.0, 3e9, False)                  # one byte short
    assert (d, j, deficit) == (OFFLOAD, i, 1.0)
    o.cancel(i)
    # deadline: t + delta <= D - now
    i = o.submit(task(TRAIN, duration=0.020, deadline=10.030))
    assert o.next(10.006, 1e12, False)[0] == IDLE               # 20 + 5 > 24 ms left
    assert o.next(10.0, 1e12, False)[:2] == (RUN, i)            # 20 + 5 <= 30 ms left


def test_foreground_first_and_yield_request():
    o = SchedOracle()
    b = o.submit(task(TRAIN, duration=0.01, utility=9.0))
    assert o.next(0.0, 1e12, False)[:2] == (RUN, b)
    assert not o.should_yield()
    f1 = o.submit(task(FOREGROUND, priority=0))
    f2 = o.submit(task(FOREGROUND, priority=5))
    assert o.should_yield()                                     # asked at its next boundary
    assert o.next(0.0, 1e12, False)[:2] == (BUSY, b)            # nothing preempts it
    o.yield_(b, True)
    assert o.next(0.0, 1e12, False)[:2] == (RUN, f2)            # higher hard priority first
    o.complete(f2, 0.001)
    assert o.next(0.0, 0.0, False)[:2] == (RUN, f1)             # no memory test for foreground
    o.complete(f1, 0.001)
    assert o.next(0.0, 1e12, False)[:2] == (RUN, b)             # the training chunk resumes


def test_no_sample_only_in_window_and_utility_order():
    o = SchedOracle()
    j = o.submit(task(JUDGE, utility=1.0))                      # no judge sample yet
    t = o.submit(task(TRAIN, duration=0.01, utility=0.5))
    assert o.next(0.0, 1e12, False)[:2] == (RUN, t)             # the judge must wait
    o.complete(t, 0.01)
    assert o.next(0.0, 1e12, False)[0] == IDLE
    assert o.next(0.0, 1e12, True)[:2] == (RUN, j)              # turn-finished window
    o.complete(j, 0.02)
    # with samples: utility decides, then priority, then arrival
    a = o.submit(task(JUDGE, utility=2.0, priority=0))
    b = o.submit(task(JUDGE, utility=2.0, priority=3))
    c = o.submit(task(JUDGE, utility=2.0, priority=3))
    assert o.next(0.0, 1e12, False)[1] == b
    o.complete(b, 0.02)
    assert o.next(0.0, 1e12, False)[1] == c
    o.complete(c, 0.02)
    assert o.next(0.0, 1e12, False)[1] == a
    # a task with no estimate is never admitted against a deadline
    o2 = SchedOracle()
    o2.submit(task(TRAIN, deadline=100.0))
    assert o2.next(0.0, 1e12, True)[0] == IDLE
