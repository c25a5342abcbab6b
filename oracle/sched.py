"""Oracle of the cooperative scheduler (test infrastructure only).

Plain Python written from the paper's §4, slow and literal: every decision
rescans every queued task. It shares nothing with the native scheduler.

§4.1 Task model. A task records (class, hard priority, adapter state,
estimated chunk duration t, estimated peak memory m, longest non-yielding
interval y, utility u). Durations come from exponential moving averages of
completed chunks: E = v for the first sample, else E = (1 - alpha) E + alpha v.
Judge and training chunks have one duration EMA each; prefill keeps a
per-token rate per prefix-length bucket b(L) in {512, 1024, ..., 32768}, and a
chunk of D tokens at prefix length L is estimated as rate[b(L)] * D.
A family with no sample yet is admitted only in an explicit turn-finished
background window.

§4.2 Foreground priority. While a foreground task is queued, no background
task starts; a background task already running is asked to stop at its next
safe boundary.

§4.3 Admission. A background task is admissible iff
    m + M_reserve <= M_free,   y + delta <= W_bg,
and, with a tool deadline D, t + delta <= D - now. The admissible task of
highest utility runs. One task runs at a time (single-task executor).

Readings where the paper is silent (also listed in the design notes):
  * foreground tasks run by hard priority, then arrival, with no memory test;
  * ties among background tasks go to the higher hard priority, then arrival;
  * a task whose duration cannot be estimated is never admitted against a
    deadline;
  * b(L) is the smallest bound >= L, the largest bound for longer prefixes;
  * with nothing admissible, if some task fails only the memory test, the
    decision is "offload": the best such task (same ranking) and the bytes it
    lacks, m + M_reserve - M_free; otherwise "idle".
"""
from __future__ import annotations

FOREGROUND, JUDGE, TRAIN, PREFILL = 0, 1, 2, 3
RUN, BUSY, IDLE, OFFLOAD = 0, 1, 2, 3
BUCKETS = (512, 1024, 2048, 4096, 8192, 16384, 32768)


def bucket(prefix_len):
    """Index of b(L)."""
    for i, bound in enumerate(BUCKETS):
        if prefix_len <= bound:
            return i
    return len(BUCKETS) - 1


class SchedOracle:
    def __init__(self, alpha_judge=0.3, alpha_train=0.3, alpha_prefill=0.3, reserve=0.0,
                 window=0.050, delta=0.005):
        self.alpha = {JUDGE: alpha_judge, TRAIN: alpha_train, PREFILL: alpha_prefill}
        self.reserve, self.window, self.delta = reserve, window, delta
        self.ema = {JUDGE: None, TRAIN: None}
        self.rate = [None] * len(BUCKETS)
        self.queue = []          # (id, task dict), in submission order
        self.next_id = 0
        self.running = None      # (id, task) or None
        self.yield_flag = False

    # ---- §4.1 estimates
    def estimate(self, task):
        if task["duration"] >= 0:
            return task["duration"]
        c = task["cls"]
        if c in (JUDGE, TRAIN):
            return -1.0 if self.ema[c] is None else self.ema[c]
        if c == PREFILL:
            r = self.rate[bucket(task["prefix_len"])]
            return -1.0 if r is None else r * task["tokens"]
        return -1.0

    def estimates(self, prefix_len):
        j = -1.0 if self.ema[JUDGE] is None else self.ema[JUDGE]
        t = -1.0 if self.ema[TRAIN] is None else self.ema[TRAIN]
        r = self.rate[bucket(prefix_len)]
        return j, t, (-1.0 if r is None else r)

    # ---- queue
    def submit(self, task):
        i = self.next_id
        self.next_id += 1
        self.queue.append((i, dict(task)))
        if task["cls"] == FOREGROUND and self.running is not None \
                and self.running[1]["cls"] != FOREGROUND:
            self.yield_flag = True
        return i

    def cancel(self, i):
        self.queue = [(j, t) for j, t in self.queue if j != i]

    # ---- §4.2 / §4.3 decision
    def next(self, now, mem_free, turn_window):
        """Returns (decision, task id or -1, estimate or -1, deficit)."""
        if self.running is not None:
            return BUSY, self.running[0], -1.0, 0.0
        fg = [(j, t) for j, t in self.queue if t["cls"] == FOREGROUND]
        if fg:
            best = fg[0]
            for j, t in fg:
                if t["priority"] > best[1]["priority"]:
                    best = (j, t)
            return self._run(best)
        admissible, short = [], []
        for j, t in self.queue:
            e = self.estimate(t)
            if e < 0:
                time_ok = bool(turn_window) and t["deadline"] < 0
            elif t["deadline"] >= 0:
                time_ok = e + self.delta <= t["deadline"] - now
            else:
                time_ok = True
            yield_ok = t["max_nonyield"] + self.delta <= self.window
            mem_ok = t["mem"] + self.reserve <= mem_free
            if time_ok and yield_ok and mem_ok:
                admissible.append((j, t))
            elif time_ok and yield_ok:
                short.append((j, t))

        def rank(jt):
            j, t = jt
            return (-t["utility"], -t["priority"], j)

        if admissible:
            return self._run(min(admissible, key=rank))
        if short:
            j, t = min(short, key=rank)
            return OFFLOAD, j, -1.0, t["mem"] + self.reserve - mem_free
        return IDLE, -1, -1.0, 0.0

    def _run(self, jt):
        j, t = jt
        self.queue = [(k, u) for k, u in self.queue if k != j]
        self.running = (j, t)
        self.yield_flag = False
        return RUN, j, self.estimate(t), 0.0

    def should_yield(self):
        return self.running is not None and self.yield_flag

    def complete(self, i, seconds):
        j, t = self.running
        assert j == i
        c = t["cls"]
        if c in (JUDGE, TRAIN):
            a = self.alpha[c]
            self.ema[c] = seconds if self.ema[c] is None else (1 - a) * self.ema[c] + a * seconds
        elif c == PREFILL and t["tokens"] > 0:
            b = bucket(t["prefix_len"])
            v = seconds / t["tokens"]
            a = self.alpha[PREFILL]
            self.rate[b] = v if self.rate[b] is None else (1 - a) * self.rate[b] + a * v
        self.running = None
        self.yield_flag = False

    def yield_(self, i, requeue):
        j, t = self.running
        assert j == i
        if requeue:  # back in its submission order
            self.queue.append((j, t))
            self.queue.sort(key=lambda jt: jt[0])
        self.running = None
        self.yield_flag = False

    def stats(self):
        n_fg = sum(1 for _, t in self.queue if t["cls"] == FOREGROUND)
        return n_fg, len(self.queue) - n_fg, (-1 if self.running is None else self.running[0])
