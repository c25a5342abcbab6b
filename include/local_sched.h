/*
 * local_sched.h — C ABI of the host-side cooperative scheduler that decides
 * which GPU-bound task runs next (§4). Nothing here touches the GPU: the
 * scheduler only admits; the caller runs what it is handed (the kernels of
 * local.h for inference and prefill, the backward for training chunks).
 *
 * It implements:
 *   - §4.1 the task model: every task records its class, hard priority,
 *     required adapter state, estimated chunk duration t, estimated peak
 *     memory m, longest non-yielding interval y and utility u. Durations are
 *     calibrated online by exponential moving averages of completed chunks:
 *     one per judge and training duration, and for prefill a per-token rate
 *     per prefix-length bucket b(L) in {512, 1024, ..., 32768}, so that the
 *     estimate of a prefill chunk of D tokens at prefix length L is
 *     rate[b(L)] * D.
 *   - §4.2 foreground priority: while a foreground task waits, no background
 *     task is admitted, and a background task that is running is asked to
 *     yield at its next safe boundary (local_sched_should_yield).
 *   - §4.3 timeslice-aware admission: with no foreground task waiting, a
 *     background task x is admissible only if
 *         m(x) + M_reserve <= M_free     and     y(x) + delta <= W_bg,
 *     and, when it carries a tool deadline D, t(x) + delta <= D - now.
 *     Among admissible tasks the one of highest utility runs. A task whose
 *     duration cannot be estimated yet (no sample of its family) is
 *     admissible only in an explicit turn-finished background window.
 *
 * Conventions
 * -----------
 *  Memory      Every pointer is HOST memory owned by the caller, except the
 *              scheduler itself (created and destroyed by the calls below).
 *  Units       Times in seconds (doubles, any origin for `now`), memory in
 *              bytes (doubles).
 *  Executor    One task runs at a time (the paper's GPU single-task
 *              executor): local_sched_next admits nothing while a task it
 *              admitted has not been reported done or yielded.
 *  Errors      Arguments are validated before anything changes; on error the
 *              scheduler is unchanged and local_last_error() (local.h) says
 *              why. Not thread-safe: one thread at a time.
 *  Determinism Every decision is a function of the call sequence alone (ties
 *              go to the higher hard priority, then the earlier submission).
 */
#ifndef LOCAL_SCHED_H
#define LOCAL_SCHED_H

#include <stdint.h>

#include "local.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct local_sched local_sched_t;

/* Task classes (§4.1). Foreground inference is the only foreground class. */
enum {
  LOCAL_TASK_FOREGROUND = 0, /* user-visible inference                            */
  LOCAL_TASK_JUDGE = 1,      /* batched judge inference (reward)                  */
  LOCAL_TASK_TRAIN = 2,      /* one training chunk up to its next commit boundary */
  LOCAL_TASK_PREFILL = 3     /* one stale-coverage or pre-prefill chunk           */
};

/* Decisions of local_sched_next. */
enum {
  LOCAL_SCHED_RUN = 0,     /* *task is admitted and now running                   */
  LOCAL_SCHED_BUSY = 1,    /* a task is running: nothing admitted                 */
  LOCAL_SCHED_IDLE = 2,    /* nothing queued, or nothing admissible               */
  LOCAL_SCHED_OFFLOAD = 3  /* nothing admissible, but some task fails only the
                              memory test: *task is the one of highest utility
                              among those, *deficit the bytes it lacks            */
};

typedef struct {
  double alpha_judge;   /* EMA weight of a new judge duration, in (0, 1]          */
  double alpha_train;   /* EMA weight of a new training-chunk duration            */
  double alpha_prefill; /* EMA weight of a new prefill per-token rate             */
  double reserve;       /* M_reserve, bytes kept for unexpected foreground work   */
  double window;        /* W_bg, the background window, seconds                   */
  double delta;         /* the conservative latency margin, seconds               */
} local_sched_params_t;

/* One task as submitted. `duration` < 0 asks the scheduler to estimate it
 * from its family's EMA (judge, training) or from the prefill rate of
 * bucket b(prefix_len) times `tokens` (prefill); foreground tasks need no
 * estimate. `deadline` < 0 means none (an absolute time otherwise).
 * mem >= 0, max_nonyield >= 0; adapter/version are recorded and returned. */
typedef struct {
  int32_t cls;          /* LOCAL_TASK_*                                           */
  int32_t priority;     /* hard priority; higher first among equal utility        */
  int32_t adapter;      /* required adapter state: adapter id ...                 */
  int32_t version;      /* ... and version                                        */
  double duration;      /* t(x), seconds, or < 0 to estimate                      */
  double mem;           /* m(x), bytes                                            */
  double max_nonyield;  /* y(x), seconds                                          */
  double utility;       /* u(x)                                                   */
  double deadline;      /* D_tool, seconds, or < 0                                */
  int32_t tokens;       /* prefill: chunk tokens D (> 0); else ignored            */
  int32_t prefix_len;   /* prefill: prefix length L (>= 0); else ignored          */
} local_sched_task_t;

/* alpha 0.3 for every family, no reserve, a 50 ms window, a 5 ms margin. */
void local_sched_default_params(local_sched_params_t* p);

/* NULL params = defaults. Fails on non-finite values, an alpha outside
 * (0, 1], or a negative reserve, window or delta. */
local_status_t local_sched_create(const local_sched_params_t* params, local_sched_t** out);
void local_sched_destroy(local_sched_t* s);

/* Queues a task; *id receives its id (ids count up from 0 in submission
 * order). A foreground task submitted while a background task runs raises
 * the yield request for that task. */
local_status_t local_sched_submit(local_sched_t* s, const local_sched_task_t* task, int64_t* id);

/* Removes a queued (not running) task. */
local_status_t local_sched_cancel(local_sched_t* s, int64_t id);

/* The admission decision at time `now` with `mem_free` bytes free.
 * `turn_window` != 0 marks an explicit turn-finished background window.
 * Foreground tasks go first (highest priority, then earliest), admitted with
 * no memory test (the reserve exists for them). Otherwise the admissible
 * background task of highest utility (ties: priority, then earliest). On
 * LOCAL_SCHED_RUN the task leaves the queue and runs; *task and, when not
 * NULL, *est (its duration estimate, -1 if unknown) are set. *deficit (may
 * be NULL) is set on LOCAL_SCHED_OFFLOAD, 0 otherwise. */
local_status_t local_sched_next(local_sched_t* s, double now, double mem_free,
                                int32_t turn_window, int32_t* decision, int64_t* task,
                                double* est, double* deficit);

/* 1 if the running task was asked to yield at its next safe boundary (a
 * foreground task arrived while it ran), else 0. */
int32_t local_sched_should_yield(const local_sched_t* s);

/* The running task finished its chunk in `seconds`: the executor is free and
 * its family's estimate takes the sample (judge, training: the duration;
 * prefill: seconds / tokens into bucket b(prefix_len); foreground: none). */
local_status_t local_sched_complete(local_sched_t* s, int64_t id, double seconds);

/* The running task stopped at a safe boundary before its chunk ended: the
 * executor is free, no sample is taken, and the task goes back to the queue
 * with its submission order (when requeue != 0) or is dropped. */
local_status_t local_sched_yield(local_sched_t* s, int64_t id, int32_t requeue);

/* Current estimates: the judge and training EMAs and the prefill rate of
 * bucket b(prefix_len); -1 where no sample exists. */
local_status_t local_sched_estimates(const local_sched_t* s, int32_t prefix_len, double* judge,
                                     double* train, double* prefill_rate);

/* Duration estimate of a prefill chunk of `tokens` at `prefix_len`
 * (rate[b(L)] * tokens), -1 if its bucket has no sample. */
local_status_t local_sched_prefill_estimate(const local_sched_t* s, int32_t tokens,
                                            int32_t prefix_len, double* seconds);

/* Queued tasks (foreground and background) and the running task id (-1). */
local_status_t local_sched_stats(const local_sched_t* s, int32_t* n_fg, int32_t* n_bg,
                                 int64_t* running);

#ifdef __cplusplus
}
#endif

#endif /* LOCAL_SCHED_H */
