// Launcher: the session plan repeated every period plus the fair,
// opportunistic, dynamic (FOD) fill of Sec. 6.1.2, run against a virtual
// integer-microsecond clock whose job durations come from the timing table.
//
// Rules (one reading of Sec. 6.1.2 and 6.3, fixed so that the outcome is a
// pure function of the table and the arrival trace):
//  - a planned job takes up to its model's batch of the oldest queued
//    requests, does not run when none are queued, and lasts its planned time;
//  - FOD runs after every arrival and every completion: candidates are the
//    models with no running job and a non-empty queue, ordered by runs in the
//    last `sessions_window` sessions, then cumulative busy time, then index
//    ("fewest runs", "least time in the GPU"); the first candidate that fits
//    starts (one per trigger) on the lowest-numbered free slots, as many as
//    its deployed share (home placement: on its home range, all of it free),
//    with the largest grid batch that is queued and whose
//    latency fits before the next planned start (at or after now) touching
//    those slots or its own next planned start;
//  - same-instant events: completions, planned starts, arrivals, each by
//    model then issue order;
//  - a served request is late if completion - arrival > SLO; no job starts
//    at or after the end of the trace, requests left queued when the last
//    started job ends are unserved; both count as violations; utilisation
//    counts slot-time inside [0, duration).
#include <algorithm>
#include <cstring>
#include <deque>
#include <map>
#include <queue>
#include <vector>

#include "sched.hpp"

namespace dstack {

namespace {

constexpr uint64_t kFnvOffset = 0xcbf29ce484222325ULL;
constexpr uint64_t kFnvPrime = 0x100000001b3ULL;

uint64_t fnv_mix(uint64_t h, int64_t v) {
  uint64_t u = (uint64_t)v;
  for (int i = 0; i < 8; ++i) {
    h ^= (u >> (8 * i)) & 0xff;
    h *= kFnvPrime;
  }
  return h;
}

struct Event {
  int64_t t;
  int kind;  // 0 completion, 1 planned start, 2 arrival
  int model;
  int64_t seq;
  uint64_t mask;
  int64_t dur;
  std::vector<int64_t> reqs;  // completion: arrival times served
  bool operator>(const Event& o) const {
    if (t != o.t) return t > o.t;
    if (kind != o.kind) return kind > o.kind;
    if (model != o.model) return model > o.model;
    return seq > o.seq;
  }
};

int64_t nearest_rank(std::vector<int64_t>& v, int pct) {
  if (v.empty()) return 0;
  std::sort(v.begin(), v.end());
  int64_t k = std::max<int64_t>(1, ((int64_t)pct * (int64_t)v.size() + 99) / 100);
  return v[(size_t)(k - 1)];
}

// latency of batch b at `slots` from the model's table: the largest swept count <= slots
int64_t table_latency(const dstack_sched_model& m, int b, int slots) {
  int row = -1;
  for (int q = 0; q < m.n_batches; ++q)
    if (m.batches[q] == b) row = q;
  if (row < 0) return -1;
  int64_t L = -1;
  for (int q = 0; q < m.n_slots; ++q)
    if (m.slots[q] <= slots && m.latency_us[row][q] > 0) L = m.latency_us[row][q];
  return L;
}

}  // namespace

dstack_status simulate(const dstack_sched_model* models, int n, const dstack_sched_params* prm,
                       const dstack_sim_params* sim, dstack_run_out* out) {
  DS_CHECK(sim && out, DSTACK_E_INVALID, "simulate: null pointer");
  DS_CHECK(sim->duration_us > 0 && sim->sessions_window >= 1, DSTACK_E_INVALID, "simulate: bad parameters");
  dstack_schedule_out* plan = new dstack_schedule_out();
  dstack_status st = schedule(models, n, prm, plan);
  if (st != DSTACK_OK && st != DSTACK_E_INFEASIBLE) {
    delete plan;
    return st;
  }
  for (int i = 0; i < n; ++i) {
    DS_CHECK(sim->n_arrivals[i] >= 0 && (sim->n_arrivals[i] == 0 || sim->arrivals_us[i]), DSTACK_E_INVALID,
             "simulate: arrivals missing");
    for (int k = 0; k < sim->n_arrivals[i]; ++k) {
      const int64_t a = sim->arrivals_us[i][k];
      DS_CHECK(a >= 0 && a < sim->duration_us && (k == 0 || a >= sim->arrivals_us[i][k - 1]), DSTACK_E_INVALID,
               "simulate: arrivals must be sorted and inside [0, duration)");
    }
  }
  const int64_t T = prm->period_us, D = sim->duration_us;
  const int total = prm->total_slots;
  const int64_t n_periods = (D + T - 1) / T;

  std::priority_queue<Event, std::vector<Event>, std::greater<Event>> ev;
  int64_t seq = 0;
  struct PStart {
    int64_t t;
    int model;
    uint64_t mask;
  };
  std::vector<PStart> pstarts;
  for (int64_t p = 0; p < n_periods; ++p)
    for (int j = 0; j < plan->n_jobs; ++j) {
      const dstack_job& job = plan->jobs[j];
      if (job.missed) continue;
      const int64_t t = p * T + job.start_us;
      if (t >= D) continue;
      Event e{t, 1, job.model, seq++, job.slot_mask, job.duration_us, {}};
      ev.push(e);
      pstarts.push_back(PStart{t, job.model, job.slot_mask});
    }
  std::sort(pstarts.begin(), pstarts.end(), [](const PStart& a, const PStart& b) { return a.t < b.t; });
  for (int i = 0; i < n; ++i)
    for (int k = 0; k < sim->n_arrivals[i]; ++k) ev.push(Event{sim->arrivals_us[i][k], 2, i, seq++, 0, 0, {}});

  std::vector<std::deque<int64_t>> queue(n);
  std::vector<char> is_running(n, 0);
  std::vector<uint64_t> run_mask(n, 0);
  uint64_t used = 0;
  std::vector<std::map<int64_t, int64_t>> runs(n);  // session -> runs
  std::vector<int64_t> busy(n, 0), served(n, 0), late(n, 0), pruns(n, 0), fruns(n, 0);
  std::vector<std::vector<int64_t>> lats(n);
  int64_t slot_us = 0, last_end = 0;
  uint64_t h = kFnvOffset;

  auto start_job = [&](int64_t t, int i, uint64_t mask, int64_t dur, int b, int kind) {
    Event c{t + dur, 0, i, seq++, mask, dur, {}};
    for (int k = 0; k < b; ++k) {
      c.reqs.push_back(queue[i].front());
      queue[i].pop_front();
    }
    is_running[i] = 1;
    run_mask[i] = mask;
    used |= mask;
    ev.push(std::move(c));
    runs[i][t / T] += 1;
    busy[i] += dur;
    slot_us += (int64_t)__builtin_popcountll(mask) * (std::min(t + dur, D) - t);  // slot-time inside [0, D)
    last_end = std::max(last_end, t + dur);
    for (int64_t v : {t, (int64_t)i, (int64_t)b, (int64_t)mask, dur, (int64_t)kind}) h = fnv_mix(h, v);
    (kind == 0 ? pruns : fruns)[i] += 1;
  };

  static const int kGrid[] = {1, 2, 4, 8, 16, 32};
  auto fod_pass = [&](int64_t t) {
    if (t >= D) return;  // nothing starts once the trace has ended
    std::vector<int> cands;
    for (int i = 0; i < n; ++i)
      if (!is_running[i] && !queue[i].empty()) cands.push_back(i);
    const int64_t cur = t / T;
    auto recent = [&](int i) {
      int64_t r = 0;
      for (auto it = runs[i].lower_bound(cur - sim->sessions_window + 1); it != runs[i].end() && it->first <= cur; ++it)
        r += it->second;
      return r;
    };
    std::stable_sort(cands.begin(), cands.end(), [&](int a, int b) {
      int64_t ra = recent(a), rb = recent(b);
      if (ra != rb) return ra < rb;
      if (busy[a] != busy[b]) return busy[a] < busy[b];
      return a < b;
    });
    for (int i : cands) {
      const int s = plan->deployed_slots[i];
      uint64_t mask = 0;
      if (prm->placement == 1) {
        mask = range_mask(plan->home_offset[i], s);
        if (used & mask) continue;
      } else {
        int got = 0;
        for (int sid = 0; sid < total && got < s; ++sid)
          if (!((used >> sid) & 1)) {
            mask |= 1ULL << sid;
            ++got;
          }
        if (got < s) continue;
      }
      // -1: no planned start constrains it; a planned start at this very
      // instant counts (same-instant planned starts are processed after
      // completions)
      int64_t gap = -1;
      for (const PStart& ps : pstarts)
        if (ps.t >= t && ((ps.mask & mask) || ps.model == i)) {
          gap = ps.t - t;
          break;
        }
      int bb = -1;
      int64_t bL = 0;
      for (int b : kGrid) {
        if (b > models[i].max_batch || b > (int)queue[i].size()) continue;
        const int64_t L = table_latency(models[i], b, s);
        if (L <= 0 || (gap >= 0 && L > gap)) continue;
        bb = b;
        bL = L;
      }
      if (bb < 0) continue;
      start_job(t, i, mask, bL, bb, 1);
      return;
    }
  };

  while (!ev.empty()) {
    Event e = ev.top();
    ev.pop();
    const int i = e.model;
    if (e.kind == 0) {
      is_running[i] = 0;
      used &= ~run_mask[i];
      for (int64_t a : e.reqs) {
        served[i] += 1;
        lats[i].push_back(e.t - a);
        if (e.t - a > models[i].slo_us) late[i] += 1;
      }
      if (sim->fod) fod_pass(e.t);
    } else if (e.kind == 1) {
      if (!queue[i].empty() && !is_running[i])
        start_job(e.t, i, e.mask, e.dur, std::min<int>(plan->batch[i], (int)queue[i].size()), 0);
    } else {
      queue[i].push_back(e.t);
      if (sim->fod) fod_pass(e.t);
    }
  }

  std::memset(out, 0, sizeof(*out));
  out->n_models = n;
  for (int i = 0; i < n; ++i) {
    dstack_model_stats& s = out->models[i];
    s.served = served[i];
    s.unserved = (int64_t)queue[i].size();
    s.violations = late[i] + s.unserved;
    s.planned_runs = pruns[i];
    s.fod_runs = fruns[i];
    s.busy_us = busy[i];
    s.p50_us = nearest_rank(lats[i], 50);
    s.p99_us = nearest_rank(lats[i], 99);
  }
  out->utilisation_ppm = (int64_t)((unsigned __int128)slot_us * 1000000 / ((unsigned __int128)total * (uint64_t)D));
  out->job_hash = h;
  out->last_end_us = last_end;
  delete plan;
  return DSTACK_OK;
}

}  // namespace dstack
