// Trajectory-task simulator (host code): a discrete-event replay of a request
// trace under one scheduling policy, with step latencies from a cost table.
// Times are int64 microseconds; the rules and policies are those stated in
// dit_sim.h.  Running steps sit in a min-heap keyed (end, request), so the
// completions at one time come out in request order; ready steps sit in
// ordered sets keyed by each policy's priority, so every dispatch decision
// costs O(log n), and each group keeps running sums of its queued work.
#include <stdarg.h>
#include <stdio.h>

#include <algorithm>
#include <functional>
#include <queue>
#include <set>
#include <string>
#include <tuple>
#include <vector>

#include "dit_sim.h"

namespace dit {
void set_last_error(const std::string& msg);
}

namespace {

dit_status sim_fail(const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  dit::set_last_error(buf);
  return DIT_ERR_INVALID_ARG;
}

struct Sim {
  // inputs
  int G, n_deg, policy, g;
  const int32_t* degrees;
  const int64_t* cost_tab;
  int64_t n;
  const int64_t* arrival;
  const int32_t* cls;
  const int32_t* n_steps;
  const int64_t* deadline;
  // per request
  std::vector<int32_t> started, done;
  std::vector<int64_t> finish, first;
  std::vector<int> bound;            // SRTF: group
  std::vector<std::vector<int>> ranks_of;  // EDF: ranks of the running step
  std::vector<int> deg_of;           // degree index of the running step
  // groups (FCFS, SRTF)
  int n_groups = 0, gk = 0;          // gk: index of the group size in degrees
  std::vector<int64_t> g_end;        // end of the running step, or -1 when idle
  std::vector<int64_t> g_queued;     // FCFS: sum of queued step costs; SRTF: sum of unstarted work
  std::vector<std::set<std::pair<int64_t, int64_t>>> fcfs_q;                   // (arrival, id)
  std::vector<std::set<std::tuple<int64_t, int64_t, int64_t>>> srtf_q;         // (work, arrival, id)
  // EDF
  std::set<std::tuple<int, int64_t, int64_t, int64_t>> edf_q;                  // (no deadline, deadline, arrival, id)
  std::set<int> free_ranks;
  // events
  typedef std::pair<int64_t, int64_t> Ev;  // (end, request)
  std::priority_queue<Ev, std::vector<Ev>, std::greater<Ev>> running;
  int64_t events = 0;
  std::vector<int64_t> dispatches;

  int64_t cost(int64_t i, int k) const { return cost_tab[(int64_t)cls[i] * n_deg + k]; }
  int64_t dl(int64_t i) const { return deadline ? deadline[i] : -1; }

  int64_t group_load(int j, int64_t now) const {
    return (g_end[j] >= 0 ? g_end[j] - now : 0) + g_queued[j];
  }

  int least_loaded(int64_t now) const {
    int best = 0;
    int64_t bl = group_load(0, now);
    for (int j = 1; j < n_groups; ++j) {
      const int64_t l = group_load(j, now);
      if (l < bl) { bl = l; best = j; }
    }
    return best;
  }

  void make_ready(int64_t i, int64_t now) {
    if (policy == DIT_SIM_FCFS_GROUPS) {
      const int j = least_loaded(now);
      fcfs_q[j].insert({arrival[i], i});
      g_queued[j] += cost(i, gk);
    } else if (policy == DIT_SIM_SRTF_GROUPS) {
      const int j = bound[i];
      srtf_q[j].insert(std::make_tuple((int64_t)(n_steps[i] - started[i]) * cost(i, gk), arrival[i], i));
    } else {
      const int64_t d = dl(i);
      edf_q.insert(std::make_tuple(d < 0 ? 1 : 0, d < 0 ? 0 : d, arrival[i], i));
    }
  }

  void start(int64_t i, int64_t now, int k) {
    if (first[i] < 0) first[i] = now;
    ++started[i];
    ++dispatches[k];
    deg_of[i] = k;
    running.push({now + cost(i, k), i});
  }

  void dispatch(int64_t now) {
    if (policy == DIT_SIM_FCFS_GROUPS) {
      for (int j = 0; j < n_groups; ++j) {
        if (g_end[j] >= 0 || fcfs_q[j].empty()) continue;
        const int64_t i = fcfs_q[j].begin()->second;
        fcfs_q[j].erase(fcfs_q[j].begin());
        g_queued[j] -= cost(i, gk);
        bound[i] = j;
        g_end[j] = now + cost(i, gk);
        start(i, now, gk);
      }
    } else if (policy == DIT_SIM_SRTF_GROUPS) {
      for (int j = 0; j < n_groups; ++j) {
        if (g_end[j] >= 0 || srtf_q[j].empty()) continue;
        const int64_t i = std::get<2>(*srtf_q[j].begin());
        srtf_q[j].erase(srtf_q[j].begin());
        g_queued[j] -= cost(i, gk);   // one unstarted step starts
        g_end[j] = now + cost(i, gk);
        start(i, now, gk);
      }
    } else {
      while (!free_ranks.empty() && !edf_q.empty()) {
        const int64_t i = std::get<3>(*edf_q.begin());
        edf_q.erase(edf_q.begin());
        const int f = (int)free_ranks.size();
        const int64_t rem = n_steps[i] - started[i];
        const int64_t d = dl(i);
        int pick = -1, fastest = 0;
        int64_t fastest_end = 0;
        for (int k = 0; k < n_deg && degrees[k] <= f; ++k) {
          const int64_t end = now + rem * cost(i, k);
          if (pick < 0 && (d < 0 || end <= d)) pick = k;
          if (k == 0 || end < fastest_end) { fastest = k; fastest_end = end; }
        }
        const int k = pick >= 0 ? pick : fastest;
        std::vector<int>& rk = ranks_of[i];
        rk.clear();
        for (int c = 0; c < degrees[k]; ++c) {
          rk.push_back(*free_ranks.begin());
          free_ranks.erase(free_ranks.begin());
        }
        start(i, now, k);
      }
    }
  }

  void run() {
    std::vector<int64_t> order(n);
    for (int64_t i = 0; i < n; ++i) order[i] = i;
    std::stable_sort(order.begin(), order.end(), [&](int64_t a, int64_t b) { return arrival[a] < arrival[b]; });
    int64_t next = 0;
    while (next < n || !running.empty()) {
      int64_t now = next < n ? arrival[order[next]] : running.top().first;
      if (!running.empty() && running.top().first < now) now = running.top().first;
      while (!running.empty() && running.top().first == now) {
        const int64_t i = running.top().second;
        running.pop();
        ++events;
        ++done[i];
        if (policy == DIT_SIM_EDF_BESTFIT) {
          for (int r : ranks_of[i]) free_ranks.insert(r);
        } else {
          g_end[bound[i]] = -1;
        }
        if (done[i] == n_steps[i]) {
          finish[i] = now;
        } else {
          make_ready(i, now);
        }
      }
      while (next < n && arrival[order[next]] == now) {
        const int64_t i = order[next++];
        ++events;
        if (policy == DIT_SIM_SRTF_GROUPS) {
          const int j = least_loaded(now);
          bound[i] = j;
          g_queued[j] += (int64_t)n_steps[i] * cost(i, gk);
        }
        make_ready(i, now);
      }
      dispatch(now);
    }
  }
};

}  // namespace

extern "C" dit_status dit_simulate(const dit_sim_config* cfg, const dit_sim_trace* tr, dit_sim_result* out) {
  dit::set_last_error("");
  if (!cfg || !tr || !out) return sim_fail("config, trace or result is NULL");
  if (cfg->n_ranks < 1) return sim_fail("n_ranks = %d", cfg->n_ranks);
  if (cfg->n_degrees < 1 || cfg->n_degrees > 16) return sim_fail("n_degrees = %d (1..16)", cfg->n_degrees);
  if (!cfg->degrees || !cfg->cost_us) return sim_fail("degrees or cost_us is NULL");
  if (cfg->degrees[0] != 1) return sim_fail("degrees[0] = %d, must be 1", cfg->degrees[0]);
  for (int k = 1; k < cfg->n_degrees; ++k)
    if (cfg->degrees[k] <= cfg->degrees[k - 1]) return sim_fail("degrees must increase strictly");
  if (cfg->n_classes < 1) return sim_fail("n_classes = %d", cfg->n_classes);
  int64_t max_cost = 0;
  for (int64_t e = 0; e < (int64_t)cfg->n_classes * cfg->n_degrees; ++e) {
    if (cfg->cost_us[e] <= 0) return sim_fail("cost_us[%lld] = %lld, must be > 0", (long long)e,
                                              (long long)cfg->cost_us[e]);
    max_cost = std::max(max_cost, cfg->cost_us[e]);
  }
  if (cfg->policy != DIT_SIM_FCFS_GROUPS && cfg->policy != DIT_SIM_SRTF_GROUPS && cfg->policy != DIT_SIM_EDF_BESTFIT)
    return sim_fail("policy %d", (int)cfg->policy);
  int gk = -1;
  if (cfg->policy != DIT_SIM_EDF_BESTFIT) {
    for (int k = 0; k < cfg->n_degrees; ++k)
      if (cfg->degrees[k] == cfg->group_size) gk = k;
    if (gk < 0) return sim_fail("group_size %d is not one of the degrees", cfg->group_size);
    if (cfg->group_size > cfg->n_ranks) return sim_fail("group_size %d > n_ranks %d", cfg->group_size, cfg->n_ranks);
  }
  if (tr->n_req < 0) return sim_fail("n_req = %lld", (long long)tr->n_req);
  if (tr->n_req > 0 && (!tr->arrival_us || !tr->cls || !tr->n_steps))
    return sim_fail("arrival_us, cls or n_steps is NULL");
  if (tr->n_req > 0 && (!out->finish_us || !out->first_start_us)) return sim_fail("finish_us or first_start_us is NULL");
  if (!out->dispatches) return sim_fail("dispatches is NULL");
  const int64_t limit = (int64_t)1 << 62;
  int64_t work = 0, last = 0;
  for (int64_t i = 0; i < tr->n_req; ++i) {
    if (tr->arrival_us[i] < 0) return sim_fail("arrival_us[%lld] < 0", (long long)i);
    if (tr->cls[i] < 0 || tr->cls[i] >= cfg->n_classes) return sim_fail("cls[%lld] = %d", (long long)i, tr->cls[i]);
    if (tr->n_steps[i] < 1) return sim_fail("n_steps[%lld] = %d", (long long)i, tr->n_steps[i]);
    last = std::max(last, tr->arrival_us[i]);
    if (last >= limit) return sim_fail("arrival_us[%lld] too large", (long long)i);
    work += (int64_t)tr->n_steps[i] * max_cost;   // n_steps < 2^31, max_cost < 2^62 / n checked below
    if (work >= limit || (int64_t)tr->n_steps[i] * max_cost >= limit)
      return sim_fail("total work exceeds 2^62 us");
  }
  if (work + last >= limit) return sim_fail("total work plus the last arrival exceeds 2^62 us");

  Sim s;
  s.G = cfg->n_ranks; s.n_deg = cfg->n_degrees; s.policy = cfg->policy; s.g = cfg->group_size;
  s.degrees = cfg->degrees; s.cost_tab = cfg->cost_us;
  s.n = tr->n_req; s.arrival = tr->arrival_us; s.cls = tr->cls; s.n_steps = tr->n_steps; s.deadline = tr->deadline_us;
  s.started.assign(s.n, 0); s.done.assign(s.n, 0);
  s.finish.assign(s.n, -1); s.first.assign(s.n, -1);
  s.bound.assign(s.n, -1); s.deg_of.assign(s.n, 0);
  s.dispatches.assign(cfg->n_degrees, 0);
  if (cfg->policy == DIT_SIM_EDF_BESTFIT) {
    s.ranks_of.resize(s.n);
    for (int r = 0; r < s.G; ++r) s.free_ranks.insert(r);
  } else {
    s.gk = gk;
    s.n_groups = s.G / s.g;
    s.g_end.assign(s.n_groups, -1);
    s.g_queued.assign(s.n_groups, 0);
    if (cfg->policy == DIT_SIM_FCFS_GROUPS) s.fcfs_q.resize(s.n_groups);
    else s.srtf_q.resize(s.n_groups);
  }
  s.run();
  for (int64_t i = 0; i < s.n; ++i) {
    out->finish_us[i] = s.finish[i];
    out->first_start_us[i] = s.first[i];
  }
  for (int k = 0; k < cfg->n_degrees; ++k) out->dispatches[k] = s.dispatches[k];
  out->events = s.events;
  return DIT_OK;
}
