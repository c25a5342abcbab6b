// Host-side cooperative scheduler (declared in local_sched.h): the task model
// with online duration estimates (§4.1), strict foreground priority with
// cooperative yield requests (§4.2) and timeslice-aware admission of
// background chunks (§4.3). Plain C++; nothing here touches the GPU.
#include <cmath>
#include <cstdint>
#include <map>

#include "../../include/local_sched.h"

local_status_t local_fail(local_status_t code, const char* fmt, ...);  // capi.hip

namespace {

constexpr int kBuckets = 7;  // prefix-length buckets 512, 1024, ..., 32768

// b(L): the smallest bucket bound >= L, the last one for longer prefixes.
int bucket_of(int32_t prefix_len) {
  int b = 0;
  int64_t bound = 512;
  while (b < kBuckets - 1 && prefix_len > bound) {
    bound *= 2;
    ++b;
  }
  return b;
}

// An exponential moving average: the first sample sets it.
struct Ema {
  bool set = false;
  double value = 0.0;
  void add(double v, double alpha) {
    value = set ? (1.0 - alpha) * value + alpha * v : v;
    set = true;
  }
  double get() const { return set ? value : -1.0; }
};

bool is_finite(double v) { return std::isfinite(v); }

}  // namespace

struct local_sched {
  local_sched_params_t p;
  Ema judge, train, rate[kBuckets];
  std::map<int64_t, local_sched_task_t> fg, bg;  // queued, by id (= submission order)
  int64_t next_id = 0;
  int64_t running = -1;
  local_sched_task_t running_task{};
  bool yield_requested = false;

  // Duration estimate of a task: its own when given, else from its family.
  double estimate(const local_sched_task_t& t) const {
    if (t.duration >= 0) return t.duration;
    switch (t.cls) {
      case LOCAL_TASK_JUDGE: return judge.get();
      case LOCAL_TASK_TRAIN: return train.get();
      case LOCAL_TASK_PREFILL: {
        const double r = rate[bucket_of(t.prefix_len)].get();
        return r < 0 ? -1.0 : r * t.tokens;
      }
      default: return -1.0;
    }
  }
};

namespace {

// Ranking of background candidates: higher utility, then higher priority,
// then earlier submission.
bool better(const local_sched_task_t& a, int64_t ia, const local_sched_task_t& b, int64_t ib) {
  if (a.utility != b.utility) return a.utility > b.utility;
  if (a.priority != b.priority) return a.priority > b.priority;
  return ia < ib;
}

}  // namespace

extern "C" void local_sched_default_params(local_sched_params_t* p) {
  if (!p) return;
  p->alpha_judge = 0.3;
  p->alpha_train = 0.3;
  p->alpha_prefill = 0.3;
  p->reserve = 0.0;
  p->window = 0.050;
  p->delta = 0.005;
}

extern "C" local_status_t local_sched_create(const local_sched_params_t* params,
                                             local_sched_t** out) {
  if (!out) return local_fail(LOCAL_ERR_NULL, "sched_create: NULL out");
  local_sched_params_t p;
  local_sched_default_params(&p);
  if (params) p = *params;
  const double alphas[3] = {p.alpha_judge, p.alpha_train, p.alpha_prefill};
  for (double a : alphas)
    if (!is_finite(a) || a <= 0.0 || a > 1.0)
      return local_fail(LOCAL_ERR_SHAPE, "sched_create: EMA weight %g outside (0, 1]", a);
  if (!is_finite(p.reserve) || !is_finite(p.window) || !is_finite(p.delta) || p.reserve < 0 ||
      p.window < 0 || p.delta < 0)
    return local_fail(LOCAL_ERR_SHAPE,
                      "sched_create: reserve %g, window %g, delta %g must be finite and >= 0",
                      p.reserve, p.window, p.delta);
  local_sched_t* s = new local_sched();
  s->p = p;
  *out = s;
  return LOCAL_OK;
}

extern "C" void local_sched_destroy(local_sched_t* s) { delete s; }

extern "C" local_status_t local_sched_submit(local_sched_t* s, const local_sched_task_t* t,
                                             int64_t* id) {
  if (!s || !t || !id) return local_fail(LOCAL_ERR_NULL, "sched_submit: NULL argument");
  if (t->cls < LOCAL_TASK_FOREGROUND || t->cls > LOCAL_TASK_PREFILL)
    return local_fail(LOCAL_ERR_SHAPE, "sched_submit: class %d", t->cls);
  if (!is_finite(t->duration) || !is_finite(t->mem) || !is_finite(t->max_nonyield) ||
      !is_finite(t->utility) || !is_finite(t->deadline) || t->mem < 0 || t->max_nonyield < 0)
    return local_fail(LOCAL_ERR_SHAPE,
                      "sched_submit: estimates must be finite, mem and max_nonyield >= 0");
  if (t->cls == LOCAL_TASK_PREFILL && t->duration < 0 && (t->tokens <= 0 || t->prefix_len < 0))
    return local_fail(LOCAL_ERR_SHAPE, "sched_submit: prefill chunk of %d tokens at %d",
                      t->tokens, t->prefix_len);
  *id = s->next_id++;
  if (t->cls == LOCAL_TASK_FOREGROUND) {
    s->fg[*id] = *t;
    if (s->running >= 0 && s->running_task.cls != LOCAL_TASK_FOREGROUND)
      s->yield_requested = true;
  } else {
    s->bg[*id] = *t;
  }
  return LOCAL_OK;
}

extern "C" local_status_t local_sched_cancel(local_sched_t* s, int64_t id) {
  if (!s) return local_fail(LOCAL_ERR_NULL, "sched_cancel: NULL scheduler");
  if (s->fg.erase(id) == 0 && s->bg.erase(id) == 0)
    return local_fail(LOCAL_ERR_SHAPE, "sched_cancel: task %lld is not queued", (long long)id);
  return LOCAL_OK;
}

extern "C" local_status_t local_sched_next(local_sched_t* s, double now, double mem_free,
                                           int32_t turn_window, int32_t* decision,
                                           int64_t* task, double* est, double* deficit) {
  if (!s || !decision || !task) return local_fail(LOCAL_ERR_NULL, "sched_next: NULL argument");
  if (!is_finite(now) || !is_finite(mem_free))
    return local_fail(LOCAL_ERR_SHAPE, "sched_next: now %g, mem_free %g", now, mem_free);
  *task = -1;
  if (est) *est = -1.0;
  if (deficit) *deficit = 0.0;
  if (s->running >= 0) {
    *decision = LOCAL_SCHED_BUSY;
    *task = s->running;
    return LOCAL_OK;
  }
  auto admit = [&](std::map<int64_t, local_sched_task_t>& q, int64_t id) {
    s->running = id;
    s->running_task = q.at(id);
    s->yield_requested = false;
    q.erase(id);
    *decision = LOCAL_SCHED_RUN;
    *task = id;
    if (est) *est = s->estimate(s->running_task);
  };
  if (!s->fg.empty()) {  // §4.2: foreground first, by hard priority, then arrival
    int64_t pick = -1;
    for (const auto& [id, t] : s->fg)
      if (pick < 0 || t.priority > s->fg.at(pick).priority) pick = id;
    admit(s->fg, pick);
    return LOCAL_OK;
  }
  // §4.3: the admissible background task of highest utility
  int64_t pick = -1, short_of_mem = -1;
  for (const auto& [id, t] : s->bg) {
    const double e = s->estimate(t);
    bool ok_time = true;
    if (e < 0) {
      // no sample of its family yet: only in a turn-finished window, and
      // never against a deadline it cannot be shown to meet
      ok_time = turn_window != 0 && t.deadline < 0;
    } else if (t.deadline >= 0) {
      ok_time = e + s->p.delta <= t.deadline - now;
    }
    const bool ok_yield = t.max_nonyield + s->p.delta <= s->p.window;
    const bool ok_mem = t.mem + s->p.reserve <= mem_free;
    if (ok_time && ok_yield && ok_mem) {
      if (pick < 0 || better(t, id, s->bg.at(pick), pick)) pick = id;
    } else if (ok_time && ok_yield) {
      if (short_of_mem < 0 || better(t, id, s->bg.at(short_of_mem), short_of_mem))
        short_of_mem = id;
    }
  }
  if (pick >= 0) {
    admit(s->bg, pick);
    return LOCAL_OK;
  }
  if (short_of_mem >= 0) {
    const local_sched_task_t& t = s->bg.at(short_of_mem);
    *decision = LOCAL_SCHED_OFFLOAD;
    *task = short_of_mem;
    if (deficit) *deficit = t.mem + s->p.reserve - mem_free;
    return LOCAL_OK;
  }
  *decision = LOCAL_SCHED_IDLE;
  return LOCAL_OK;
}

extern "C" int32_t local_sched_should_yield(const local_sched_t* s) {
  return (s && s->running >= 0 && s->yield_requested) ? 1 : 0;
}

extern "C" local_status_t local_sched_complete(local_sched_t* s, int64_t id, double seconds) {
  if (!s) return local_fail(LOCAL_ERR_NULL, "sched_complete: NULL scheduler");
  if (id < 0 || id != s->running)
    return local_fail(LOCAL_ERR_SHAPE, "sched_complete: task %lld is not running",
                      (long long)id);
  if (!is_finite(seconds) || seconds < 0)
    return local_fail(LOCAL_ERR_SHAPE, "sched_complete: duration %g", seconds);
  const local_sched_task_t& t = s->running_task;
  switch (t.cls) {
    case LOCAL_TASK_JUDGE: s->judge.add(seconds, s->p.alpha_judge); break;
    case LOCAL_TASK_TRAIN: s->train.add(seconds, s->p.alpha_train); break;
    case LOCAL_TASK_PREFILL:
      if (t.tokens > 0)
        s->rate[bucket_of(t.prefix_len)].add(seconds / t.tokens, s->p.alpha_prefill);
      break;
    default: break;
  }
  s->running = -1;
  s->yield_requested = false;
  return LOCAL_OK;
}

extern "C" local_status_t local_sched_yield(local_sched_t* s, int64_t id, int32_t requeue) {
  if (!s) return local_fail(LOCAL_ERR_NULL, "sched_yield: NULL scheduler");
  if (id < 0 || id != s->running)
    return local_fail(LOCAL_ERR_SHAPE, "sched_yield: task %lld is not running", (long long)id);
  if (requeue) {
    if (s->running_task.cls == LOCAL_TASK_FOREGROUND)
      s->fg[id] = s->running_task;
    else
      s->bg[id] = s->running_task;
  }
  s->running = -1;
  s->yield_requested = false;
  return LOCAL_OK;
}

extern "C" local_status_t local_sched_estimates(const local_sched_t* s, int32_t prefix_len,
                                                double* judge, double* train,
                                                double* prefill_rate) {
  if (!s || !judge || !train || !prefill_rate)
    return local_fail(LOCAL_ERR_NULL, "sched_estimates: NULL argument");
  *judge = s->judge.get();
  *train = s->train.get();
  *prefill_rate = s->rate[bucket_of(prefix_len)].get();
  return LOCAL_OK;
}

extern "C" local_status_t local_sched_prefill_estimate(const local_sched_t* s, int32_t tokens,
                                                       int32_t prefix_len, double* seconds) {
  if (!s || !seconds) return local_fail(LOCAL_ERR_NULL, "sched_prefill_estimate: NULL argument");
  if (tokens <= 0 || prefix_len < 0)
    return local_fail(LOCAL_ERR_SHAPE, "sched_prefill_estimate: %d tokens at %d", tokens,
                      prefix_len);
  const double r = s->rate[bucket_of(prefix_len)].get();
  *seconds = r < 0 ? -1.0 : r * tokens;
  return LOCAL_OK;
}

extern "C" local_status_t local_sched_stats(const local_sched_t* s, int32_t* n_fg,
                                            int32_t* n_bg, int64_t* running) {
  if (!s || !n_fg || !n_bg || !running)
    return local_fail(LOCAL_ERR_NULL, "sched_stats: NULL argument");
  *n_fg = static_cast<int32_t>(s->fg.size());
  *n_bg = static_cast<int32_t>(s->bg.size());
  *running = s->running;
  return LOCAL_OK;
}
