// Load-aware scheduler of the offloading engine (Sec. 3.2) and its cost model,
// as a discrete-time simulator over per-layer stage times.
//
// Cost model (Sec. 3.2): per-layer times of GPU decode attention T_ga and CPU
// decode attention T_ca are profiled offline on a grid of (requests, total
// context tokens) and linearly interpolated (bilinear inside the grid, the
// edge cell's plane outside it); the linear stage T_l (pre- plus
// post-projection) is a curve over the sub-batch's token count. The
// iteration time of a two-batch schedule is
//   T = L * (max(T_l0, T_ca1) + max(T_l1 + T_ga0, T_ca0)),
// and of a GPU-only schedule L * (T_l0 + T_ga0).
//
// Each step() makes one iteration's schedule in the paper's six steps
// (initialise; GPU decodes with swap-out / swap-in; prefills; CPU decodes
// under T_ca1 <= T_l0 and T_ca0 <= T_l1 + T_ga0; removal of prefills whose
// KV would be swapped out; greedy choice between the two-batch and the
// GPU-only schedule by estimated throughput) and then advances every
// scheduled request by one token. Host C++, no GPU.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <deque>
#include <new>
#include <vector>

#include "libneoattn.h"
#include "neo_error.h"

namespace neo {
namespace sched {
namespace {

struct Grid {
  std::vector<double> b, s, t;  // t[i * s.size() + j]
};

struct Curve {
  std::vector<double> x, t;
};

// Index of the cell [v[i], v[i+1]] used for x: the last one whose left end is
// <= x, clamped to the first / last cell (so outside the axis the edge cell's
// line extends). -1 when the axis has one point.
int cell(const std::vector<double>& v, double x) {
  const int n = (int)v.size();
  if (n < 2) return -1;
  int i = (int)(std::upper_bound(v.begin(), v.end(), x) - v.begin()) - 1;
  return std::min(std::max(i, 0), n - 2);
}

// Position of x in cell i as a fraction (may be < 0 or > 1 outside the axis).
double frac(const std::vector<double>& v, int i, double x) {
  return (x - v[i]) / (v[i + 1] - v[i]);
}

double eval_curve(const Curve& c, double x) {
  const int i = cell(c.x, x);
  if (i < 0) return c.t[0];
  const double u = frac(c.x, i, x);
  return c.t[i] + u * (c.t[i + 1] - c.t[i]);
}

double eval_grid(const Grid& g, double b, double s) {
  const int ns = (int)g.s.size();
  const int i = cell(g.b, b), j = cell(g.s, s);
  const double u = i < 0 ? 0.0 : frac(g.b, i, b);
  const double v = j < 0 ? 0.0 : frac(g.s, j, s);
  const int i0 = i < 0 ? 0 : i, i1 = i < 0 ? 0 : i + 1;
  const int j0 = j < 0 ? 0 : j, j1 = j < 0 ? 0 : j + 1;
  const double t00 = g.t[i0 * ns + j0], t01 = g.t[i0 * ns + j1];
  const double t10 = g.t[i1 * ns + j0], t11 = g.t[i1 * ns + j1];
  const double lo = t00 + v * (t01 - t00);  // along s at b = b[i0]
  const double hi = t10 + v * (t11 - t10);  // along s at b = b[i1]
  return lo + u * (hi - lo);
}

neo_status check_axis(const double* v, int32_t n, const char* what) {
  if (n < 1 || !v) return set_error(NEO_ERR_INVALID_ARG, "%s: empty axis", what);
  for (int32_t i = 0; i < n; ++i) {
    if (!std::isfinite(v[i])) return set_error(NEO_ERR_INVALID_ARG, "%s: non-finite value", what);
    if (i > 0 && !(v[i] > v[i - 1]))
      return set_error(NEO_ERR_INVALID_ARG, "%s: axis not strictly ascending", what);
  }
  return NEO_OK;
}

neo_status load_grid(const neo_cost_grid& in, Grid* out, const char* what) {
  neo_status st = check_axis(in.b, in.n_b, what);
  if (st != NEO_OK) return st;
  st = check_axis(in.s, in.n_s, what);
  if (st != NEO_OK) return st;
  if (!in.t) return set_error(NEO_ERR_INVALID_ARG, "%s: no times", what);
  out->b.assign(in.b, in.b + in.n_b);
  out->s.assign(in.s, in.s + in.n_s);
  out->t.assign(in.t, in.t + (size_t)in.n_b * in.n_s);
  for (double t : out->t)
    if (!std::isfinite(t)) return set_error(NEO_ERR_INVALID_ARG, "%s: non-finite time", what);
  return NEO_OK;
}

neo_status load_curve(const neo_cost_curve& in, Curve* out, const char* what) {
  neo_status st = check_axis(in.x, in.n, what);
  if (st != NEO_OK) return st;
  if (!in.t) return set_error(NEO_ERR_INVALID_ARG, "%s: no times", what);
  out->x.assign(in.x, in.x + in.n);
  out->t.assign(in.t, in.t + in.n);
  for (double t : out->t)
    if (!std::isfinite(t)) return set_error(NEO_ERR_INVALID_ARG, "%s: non-finite time", what);
  return NEO_OK;
}

enum Where : int8_t { kFuture, kWaiting, kGpu, kCpu, kDone };

struct Req {
  int64_t id;
  int32_t prompt, output;
  double arrival;
  int64_t ctx = 0;          // tokens whose KV is cached
  int64_t generated = 0;    // output tokens produced so far
  int64_t prefill_len = 0;  // tokens the next prefill computes
  Where where = kFuture;
};

}  // namespace

struct Scheduler {
  neo_sched_config cfg{};
  Grid t_ga, t_ca;
  Curve t_l;
  std::vector<Req> reqs;
  std::vector<int> arrivals;  // indices sorted by (arrival, id), not yet arrived
  size_t next_arrival = 0;
  bool sorted = true;
  std::deque<int> waitq;       // prefill wait queue (FIFO)
  std::vector<int> gpu_run;    // GPU decoding run queue, in admission order
  std::vector<int> cpu_run;    // CPU decoding run queue, in admission order
  int64_t cpu_held = 0;        // blocks held in the CPU cache
  double now = 0.0;
  int64_t tokens = 0, iterations = 0, finished = 0, two_batch_iters = 0;
  int64_t swapped_out = 0, swapped_in = 0, preempted = 0;

  int64_t blocks(int64_t tokens_) const { return (tokens_ + cfg.block_size - 1) / cfg.block_size; }

  double tl(int64_t x) const { return x <= 0 ? 0.0 : eval_curve(t_l, (double)x); }
  double tga(int64_t n, int64_t s) const { return n <= 0 ? 0.0 : eval_grid(t_ga, (double)n, (double)s); }
  double tca(int64_t n, int64_t s) const { return n <= 0 ? 0.0 : eval_grid(t_ca, (double)n, (double)s); }

  void admit_arrivals() {
    if (!sorted) {
      std::stable_sort(arrivals.begin() + next_arrival, arrivals.end(), [&](int a, int b) {
        return reqs[a].arrival < reqs[b].arrival ||
               (reqs[a].arrival == reqs[b].arrival && reqs[a].id < reqs[b].id);
      });
      sorted = true;
    }
    while (next_arrival < arrivals.size() && reqs[arrivals[next_arrival]].arrival <= now) {
      Req& r = reqs[arrivals[next_arrival++]];
      r.where = kWaiting;
      r.prefill_len = r.prompt;
      waitq.push_back((int)(&r - reqs.data()));
    }
  }

  void finish(Req& r) {
    r.where = kDone;
    ++finished;
  }

  neo_status step(neo_sched_iter* info, int64_t* ids, int64_t cap);
};

neo_status Scheduler::step(neo_sched_iter* info, int64_t* ids, int64_t cap) {
  admit_arrivals();
  *info = neo_sched_iter{};
  if (waitq.empty() && gpu_run.empty() && cpu_run.empty()) {
    if (next_arrival >= arrivals.size()) {
      info->done = 1;
      return NEO_OK;
    }
    now = std::max(now, reqs[arrivals[next_arrival]].arrival);  // idle until the next arrival
    admit_arrivals();
  }

  // Step 1: two empty sub-batches.
  std::vector<int> pre, gpu_dec, cpu0, cpu1, sw_out, sw_in;
  std::vector<char> pre_swap;  // per prefill: its KV goes to the CPU cache

  // Step 2: every GPU decoding request into batch-0; swap out (most recently
  // admitted first) until the GPU cache holds every request's next token; a
  // request the CPU cache cannot take either is preempted (recomputed later).
  int64_t gpu_need = 0;
  for (int i : gpu_run) gpu_need += blocks(reqs[i].ctx + 1);
  while (gpu_need > cfg.gpu_blocks && !gpu_run.empty()) {
    const int i = gpu_run.back();
    gpu_run.pop_back();
    Req& r = reqs[i];
    gpu_need -= blocks(r.ctx + 1);
    if (cpu_held + blocks(r.ctx) <= cfg.cpu_blocks) {
      r.where = kCpu;
      cpu_held += blocks(r.ctx);
      cpu_run.push_back(i);
      sw_out.push_back(i);
      ++swapped_out;
    } else {
      r.where = kWaiting;
      r.prefill_len = r.ctx;
      r.ctx = 0;
      waitq.push_front(i);
      ++preempted;
    }
  }
  gpu_dec = gpu_run;
  // Swap in (oldest CPU request first) while the GPU cache keeps
  // swap_in_reserve_blocks free after the move (no reserve while the GPU runs
  // nothing: it only leaves room for running requests to grow).
  {
    size_t k = 0;
    const bool fresh = sw_out.empty();  // never swap back what was just swapped out
    while (fresh && k < cpu_run.size()) {
      const int i = cpu_run[k];
      Req& r = reqs[i];
      const int64_t reserve = gpu_run.empty() ? 0 : cfg.swap_in_reserve_blocks;
      if (gpu_need + blocks(r.ctx + 1) + reserve > cfg.gpu_blocks) break;
      gpu_need += blocks(r.ctx + 1);
      cpu_held -= blocks(r.ctx);
      r.where = kGpu;
      cpu_run.erase(cpu_run.begin() + k);
      gpu_run.push_back(i);
      gpu_dec.push_back(i);
      sw_in.push_back(i);
      ++swapped_in;
    }
  }

  // Step 3: prefills from the wait queue into batch-0 while the GPU can hold
  // the batch's activations; their KV stays on the GPU if the GPU cache has
  // room, else it is swapped out to the CPU cache as it is produced.
  int64_t act0 = (int64_t)gpu_dec.size();  // tokens of batch-0's linear stage
  int64_t cpu_plan = cpu_held;             // CPU blocks after this iteration's placements
  while (!waitq.empty()) {
    const int i = waitq.front();
    const Req& r = reqs[i];
    // (A prompt longer than the activation limit still runs alone.)
    if (act0 > 0 && act0 + r.prefill_len > cfg.max_batch_tokens) break;
    const int64_t nb = blocks(r.prefill_len);
    if (gpu_need + nb <= cfg.gpu_blocks) {
      gpu_need += nb;
      pre_swap.push_back(0);
    } else if (cpu_plan + nb <= cfg.cpu_blocks) {
      cpu_plan += nb;
      pre_swap.push_back(1);
    } else {
      break;
    }
    waitq.pop_front();
    pre.push_back(i);
    act0 += r.prefill_len;
  }

  // Step 4: CPU decoding requests into batch-1 (tried first) or batch-0,
  // keeping T_ca1 <= T_l0 and T_ca0 <= T_l1 + T_ga0; a request that fits
  // neither waits for the next iteration.
  int64_t s_ga0 = 0;
  for (int i : gpu_dec) s_ga0 += reqs[i].ctx + 1;
  const double t_ga0 = tga((int64_t)gpu_dec.size(), s_ga0);
  int64_t s_ca0 = 0, s_ca1 = 0;
  double t_ca0 = 0.0, t_ca1 = 0.0;
  double t_l0 = tl(act0), t_l1 = 0.0;
  if (cfg.policy == NEO_SCHED_POLICY_NEO) {
    for (int i : cpu_run) {
      const Req& r = reqs[i];
      const int64_t grow = blocks(r.ctx + 1) - blocks(r.ctx);
      if (cpu_plan + grow > cfg.cpu_blocks) continue;
      if (act0 + (int64_t)cpu1.size() + 1 > cfg.max_batch_tokens) break;
      const int64_t len = r.ctx + 1;
      const double ca1 = tca((int64_t)cpu1.size() + 1, s_ca1 + len);
      const double l1 = tl((int64_t)cpu1.size() + 1);
      if (ca1 <= t_l0 && t_ca0 <= l1 + t_ga0) {
        cpu1.push_back(i);
        s_ca1 += len;
        t_ca1 = ca1;
        t_l1 = l1;
        cpu_plan += grow;
        continue;
      }
      const double ca0 = tca((int64_t)cpu0.size() + 1, s_ca0 + len);
      const double l0 = tl(act0 + 1);
      if (ca0 <= t_l1 + t_ga0 && t_ca1 <= l0) {
        cpu0.push_back(i);
        s_ca0 += len;
        t_ca0 = ca0;
        t_l0 = l0;
        ++act0;
        cpu_plan += grow;
      }
    }

    // Step 5: while batch-1 gives the CPU work, drop prefills whose KV would
    // be swapped out (latest first) as long as both inequalities still hold.
    if (!cpu1.empty()) {
      for (int k = (int)pre.size() - 1; k >= 0; --k) {
        if (!pre_swap[k]) continue;
        const Req& r = reqs[pre[k]];
        const double l0 = tl(act0 - r.prefill_len);
        if (t_ca1 <= l0 && t_ca0 <= t_l1 + t_ga0) {
          act0 -= r.prefill_len;
          t_l0 = l0;
          cpu_plan -= blocks(r.prefill_len);
          waitq.push_front(pre[k]);
          pre.erase(pre.begin() + k);
          pre_swap.erase(pre_swap.begin() + k);
        }
      }
    }
  }

  // Progress: an iteration that would run nothing while requests wait on
  // the CPU (the GPU holds none of them and none can move there) runs them on
  // the CPU without the balance constraints.
  if (cfg.policy == NEO_SCHED_POLICY_NEO && pre.empty() && gpu_dec.empty() && cpu0.empty() &&
      cpu1.empty()) {
    for (int i : cpu_run) {
      const Req& r = reqs[i];
      const int64_t grow = blocks(r.ctx + 1) - blocks(r.ctx);
      if (cpu_plan + grow > cfg.cpu_blocks) continue;
      if ((int64_t)cpu1.size() + 1 > cfg.max_batch_tokens) break;
      cpu1.push_back(i);
      s_ca1 += r.ctx + 1;
      cpu_plan += grow;
    }
    t_ca1 = tca((int64_t)cpu1.size(), s_ca1);
    t_l1 = tl((int64_t)cpu1.size());
  }
  if (pre.empty() && gpu_dec.empty() && cpu0.empty() && cpu1.empty())
    return set_error(NEO_ERR_INVALID_ARG,
                     "nothing can be scheduled: a waiting request fits neither cache");

  // Step 6: the GPU-only schedule is batch-0 without its CPU decodes; keep
  // the schedule with the higher estimated throughput x / T (compared as
  // x_two * T_gpu > x_gpu * T_two).
  const double L = (double)cfg.num_layers;
  const double t_two = L * (std::max(t_l0, t_ca1) + std::max(t_l1 + t_ga0, t_ca0));
  const int64_t act_gpu = act0 - (int64_t)cpu0.size();
  const double t_gpu = L * (tl(act_gpu) + t_ga0);
  const int64_t x_two = (int64_t)(pre.size() + gpu_dec.size() + cpu0.size() + cpu1.size());
  const int64_t x_gpu = (int64_t)(pre.size() + gpu_dec.size());
  bool two;
  if (cpu0.empty() && cpu1.empty())
    two = false;
  else if (x_gpu == 0)
    two = true;
  else
    two = (double)x_two * t_gpu > (double)x_gpu * t_two;
  const double t_iter = two ? t_two : t_gpu;

  // Report.
  info->mode = two ? NEO_SCHED_TWO_BATCH : NEO_SCHED_GPU_ONLY;
  info->t_iter = t_iter;
  info->t_two_batch = t_two;
  info->t_gpu_only = t_gpu;
  info->t_l0 = t_l0;
  info->t_l1 = t_l1;
  info->t_ga0 = t_ga0;
  info->t_ca0 = t_ca0;
  info->t_ca1 = t_ca1;
  info->n_prefill = (int32_t)pre.size();
  info->n_gpu_decode = (int32_t)gpu_dec.size();
  info->n_cpu_decode0 = two ? (int32_t)cpu0.size() : 0;
  info->n_cpu_decode1 = two ? (int32_t)cpu1.size() : 0;
  info->n_swap_out = (int32_t)sw_out.size();
  info->n_swap_in = (int32_t)sw_in.size();
  info->n_prefill_to_cpu = 0;
  for (char c : pre_swap) info->n_prefill_to_cpu += c;
  const int64_t nids = (int64_t)pre.size() + (int64_t)gpu_dec.size() + info->n_cpu_decode0 +
                       info->n_cpu_decode1 + (int64_t)sw_out.size() + (int64_t)sw_in.size();
  if (ids) {
    if (cap < nids)
      return set_error(NEO_ERR_INVALID_ARG, "ids capacity %lld < %lld needed", (long long)cap,
                       (long long)nids);
  }
  int64_t w = 0;
  auto put = [&](const std::vector<int>& v) {
    for (int i : v) {
      if (ids) ids[w] = reqs[i].id;
      ++w;
    }
  };
  put(pre);
  put(gpu_dec);
  if (two) {
    put(cpu0);
    put(cpu1);
  }
  put(sw_out);
  put(sw_in);

  // Advance: every scheduled request produces one token.
  std::vector<int> done_gpu;
  for (size_t k = 0; k < pre.size(); ++k) {
    Req& r = reqs[pre[k]];
    r.ctx = r.prefill_len;
    r.generated += 1;
    if (r.generated >= r.output) {
      if (pre_swap[k]) cpu_plan -= blocks(r.ctx);
      finish(r);
    } else if (pre_swap[k]) {
      r.where = kCpu;
      cpu_run.push_back(pre[k]);
    } else {
      r.where = kGpu;
      gpu_run.push_back(pre[k]);
    }
  }
  auto decode = [&](int i, bool on_cpu) {
    Req& r = reqs[i];
    r.ctx += 1;
    r.generated += 1;
    if (r.generated >= r.output) {
      if (on_cpu) cpu_plan -= blocks(r.ctx);
      finish(r);
      return true;
    }
    return false;
  };
  for (int i : gpu_dec) decode(i, false);
  gpu_run.erase(std::remove_if(gpu_run.begin(), gpu_run.end(),
                               [&](int i) { return reqs[i].where == kDone; }),
                gpu_run.end());
  if (two) {
    for (int i : cpu0) decode(i, true);
    for (int i : cpu1) decode(i, true);
  } else {
    // CPU decodes were not run: give back their planned growth.
    for (int i : cpu0) cpu_plan -= blocks(reqs[i].ctx + 1) - blocks(reqs[i].ctx);
    for (int i : cpu1) cpu_plan -= blocks(reqs[i].ctx + 1) - blocks(reqs[i].ctx);
  }
  cpu_run.erase(std::remove_if(cpu_run.begin(), cpu_run.end(),
                               [&](int i) { return reqs[i].where == kDone; }),
                cpu_run.end());
  cpu_held = cpu_plan;

  now += t_iter;
  tokens += two ? x_two : x_gpu;
  iterations += 1;
  two_batch_iters += two ? 1 : 0;
  info->n_tokens = two ? x_two : x_gpu;
  info->now = now;
  return NEO_OK;
}

}  // namespace sched
}  // namespace neo

struct neo_sched {
  neo::sched::Scheduler s;
};

extern "C" {

neo_status neo_cost_eval_grid(const neo_cost_grid* grid, double b, double s, double* out) {
  using namespace neo::sched;
  if (!grid || !out) return neo::set_error(NEO_ERR_INVALID_ARG, "a required pointer is NULL");
  Grid g;
  neo_status st = load_grid(*grid, &g, "grid");
  if (st != NEO_OK) return st;
  *out = eval_grid(g, b, s);
  return neo::clear_error();
}

neo_status neo_cost_eval_curve(const neo_cost_curve* curve, double x, double* out) {
  using namespace neo::sched;
  if (!curve || !out) return neo::set_error(NEO_ERR_INVALID_ARG, "a required pointer is NULL");
  Curve c;
  neo_status st = load_curve(*curve, &c, "curve");
  if (st != NEO_OK) return st;
  *out = eval_curve(c, x);
  return neo::clear_error();
}

neo_status neo_sched_create(const neo_sched_config* cfg, neo_sched** out) {
  using namespace neo::sched;
  if (!cfg || !out) return neo::set_error(NEO_ERR_INVALID_ARG, "a required pointer is NULL");
  *out = nullptr;
  if (cfg->num_layers <= 0 || cfg->block_size <= 0)
    return neo::set_error(NEO_ERR_INVALID_ARG, "num_layers and block_size must be positive");
  if (cfg->gpu_blocks < 0 || cfg->cpu_blocks < 0 || cfg->max_batch_tokens <= 0 ||
      cfg->swap_in_reserve_blocks < 0)
    return neo::set_error(NEO_ERR_INVALID_ARG, "capacities must be non-negative (max_batch_tokens positive)");
  if (cfg->policy != NEO_SCHED_POLICY_NEO && cfg->policy != NEO_SCHED_POLICY_GPU_ONLY)
    return neo::set_error(NEO_ERR_UNSUPPORTED, "policy %d unknown", cfg->policy);
  neo_sched* s = new (std::nothrow) neo_sched();
  if (!s) return neo::set_error(NEO_ERR_INVALID_ARG, "out of host memory");
  s->s.cfg = *cfg;
  neo_status st = load_grid(cfg->t_ga, &s->s.t_ga, "t_ga");
  if (st == NEO_OK) st = load_grid(cfg->t_ca, &s->s.t_ca, "t_ca");
  if (st == NEO_OK) st = load_curve(cfg->t_l, &s->s.t_l, "t_l");
  if (st != NEO_OK) {
    delete s;
    return st;
  }
  // The tables are copied; the config's pointers are not kept.
  s->s.cfg.t_ga = neo_cost_grid{};
  s->s.cfg.t_ca = neo_cost_grid{};
  s->s.cfg.t_l = neo_cost_curve{};
  *out = s;
  return neo::clear_error();
}

neo_status neo_sched_add_request(neo_sched* s, int64_t id, int32_t prompt_len, int32_t output_len,
                                 double arrival) {
  if (!s) return neo::set_error(NEO_ERR_INVALID_ARG, "scheduler is NULL");
  if (prompt_len <= 0 || output_len <= 0)
    return neo::set_error(NEO_ERR_INVALID_ARG, "prompt_len and output_len must be positive");
  if (!std::isfinite(arrival) || arrival < 0)
    return neo::set_error(NEO_ERR_INVALID_ARG, "arrival must be finite and >= 0");
  neo::sched::Req r;
  r.id = id;
  r.prompt = prompt_len;
  r.output = output_len;
  r.arrival = std::max(arrival, s->s.now);
  s->s.reqs.push_back(r);
  s->s.arrivals.push_back((int)s->s.reqs.size() - 1);
  s->s.sorted = false;
  return neo::clear_error();
}

neo_status neo_sched_step(neo_sched* s, neo_sched_iter* info, int64_t* ids, int64_t ids_capacity) {
  if (!s || !info) return neo::set_error(NEO_ERR_INVALID_ARG, "a required pointer is NULL");
  neo_status st = s->s.step(info, ids, ids_capacity);
  if (st != NEO_OK) return st;
  return neo::clear_error();
}

neo_status neo_sched_get_stats(const neo_sched* s, neo_sched_stats* out) {
  if (!s || !out) return neo::set_error(NEO_ERR_INVALID_ARG, "a required pointer is NULL");
  const auto& x = s->s;
  out->now = x.now;
  out->tokens = x.tokens;
  out->iterations = x.iterations;
  out->two_batch_iterations = x.two_batch_iters;
  out->finished = x.finished;
  out->swapped_out = x.swapped_out;
  out->swapped_in = x.swapped_in;
  out->preempted = x.preempted;
  int64_t gpu = 0;
  for (int i : x.gpu_run) gpu += x.blocks(x.reqs[i].ctx);
  out->gpu_blocks_held = gpu;
  out->cpu_blocks_held = x.cpu_held;
  out->waiting = (int64_t)x.waitq.size();
  out->gpu_running = (int64_t)x.gpu_run.size();
  out->cpu_running = (int64_t)x.cpu_run.size();
  return neo::clear_error();
}

void neo_sched_destroy(neo_sched* s) { delete s; }

}  // extern "C"
