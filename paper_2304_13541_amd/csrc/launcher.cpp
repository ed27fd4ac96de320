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
#include "launcher.hpp"

#include <algorithm>
#include <cstring>
#include <queue>

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

const int kGrid[] = {1, 2, 4, 8, 16, 32};

}  // namespace

int64_t nearest_rank(std::vector<int64_t>& v, int pct) {
  if (v.empty()) return 0;
  std::sort(v.begin(), v.end());
  int64_t k = std::max<int64_t>(1, ((int64_t)pct * (int64_t)v.size() + 99) / 100);
  return v[(size_t)(k - 1)];
}

bool check_trace(int n, const dstack_sim_params* sim) {
  if (sim->duration_us <= 0 || sim->sessions_window < 1 || sim->policy < 0 || sim->policy > 3 ||
      sim->slice_cycle_us < 0 || sim->resize_violations < 0)
    return false;
  for (int i = 0; i < n; ++i) {
    if (sim->n_arrivals[i] < 0 || (sim->n_arrivals[i] > 0 && !sim->arrivals_us[i])) return false;
    for (int k = 0; k < sim->n_arrivals[i]; ++k) {
      const int64_t a = sim->arrivals_us[i][k];
      if (a < 0 || a >= sim->duration_us || (k > 0 && a < sim->arrivals_us[i][k - 1])) return false;
    }
  }
  return true;
}

LaunchState::LaunchState(const dstack_sched_model* models, int n, const dstack_sched_params* prm,
                         const dstack_sim_params* sim, const dstack_schedule_out* plan)
    : models_(models), n_(n), prm_(prm), sim_(sim), plan_(plan), T_(prm->period_us), D_(sim->duration_us),
      queue_(n), running_(n, 0), run_mask_(n, 0), runs_(n), busy_(n, 0), dep_(n), home_(n), viol_(n, 0),
      resizes_(n, 0), changed_at_(n, 0), avail_(n, 1) {
  for (int i = 0; i < n; ++i) {
    dep_[i] = plan->deployed_slots[i];
    home_[i] = prm->placement == 1 ? plan->home_offset[i] : 0;
  }
  const int64_t n_periods = sim->policy == 0 ? (D_ + T_ - 1) / T_ : 0;  // the comparators run no plan
  for (int64_t p = 0; p < n_periods; ++p)
    for (int j = 0; j < plan->n_jobs; ++j) {
      const dstack_job& job = plan->jobs[j];
      if (job.missed) continue;
      const int64_t t = p * T_ + job.start_us;
      if (t < D_) pstarts_.push_back(PlannedStart{t, job.model, job.slot_mask, job.duration_us});
    }
  std::stable_sort(pstarts_.begin(), pstarts_.end(),
                   [](const PlannedStart& a, const PlannedStart& b) { return a.t < b.t; });
  if (sim->policy == 3) {  // temporal: slices proportional to the SLOs, repeated every cycle
    int64_t slo_min = models[0].slo_us, slo_sum = 0;
    for (int i = 0; i < n; ++i) {
      slo_min = std::min(slo_min, models[i].slo_us);
      slo_sum += models[i].slo_us;
    }
    cycle_ = sim->slice_cycle_us > 0 ? sim->slice_cycle_us : slo_min;
    int64_t off = 0;
    for (int i = 0; i < n; ++i) {
      const int64_t len = (int64_t)((unsigned __int128)cycle_ * (uint64_t)models[i].slo_us / (uint64_t)slo_sum);
      slice_off_.push_back(off);
      slice_len_.push_back(len);
      off += len;
    }
    const uint64_t all = range_mask(0, prm->total_slots);
    for (int64_t k = 0; k * cycle_ < D_; ++k)
      for (int i = 0; i < n; ++i) {
        const int64_t t = k * cycle_ + slice_off_[i];
        if (slice_len_[i] > 0 && t < D_) slices_.push_back(PlannedStart{t, i, all, 0});
      }
  }
}

bool LaunchState::note_late(int64_t t, int i, int64_t late) {
  if (sim_->policy != 0 || sim_->resize_violations <= 0) return false;
  viol_[i] += late;
  if (viol_[i] < sim_->resize_violations) return false;
  viol_[i] = 0;
  int home = 0, next = 0;
  if (!next_range(i, &home, &next)) return false;  // already at its largest swept share
  dep_[i] = next;
  home_[i] = home;
  resizes_[i] += 1;
  changed_at_[i] = t;
  return true;
}

int64_t LaunchState::late_at_end(int i, int64_t start, int64_t end, const std::vector<int64_t>& reqs) const {
  int64_t c = 0;
  for (int64_t a : reqs)
    if (a >= changed_at_[i] && end - a > models_[i].slo_us && 2 * (start - a) <= models_[i].slo_us) c += 1;
  return c;
}

bool LaunchState::next_range(int i, int* home, int* dep) const {
  const dstack_sched_model& m = models_[i];
  int next = -1;
  for (int q = 0; q < m.n_slots && next < 0; ++q)
    if (m.slots[q] > dep_[i] && m.slots[q] <= prm_->total_slots && table_latency(i, plan_->batch[i], m.slots[q]) > 0)
      next = m.slots[q];
  if (next < 0) return false;
  const int h = home_[i] + next > prm_->total_slots ? prm_->total_slots - next : home_[i];
  // no change that would make the model contend with one whose range its
  // current range does not meet
  const uint64_t now = range_mask(home_[i], dep_[i]), grown = range_mask(h, next);
  for (int j = 0; j < n_; ++j) {
    if (j == i) continue;
    const uint64_t other = range_mask(home_[j], dep_[j]);
    if ((grown & other) && !(now & other)) return false;
  }
  *dep = next;
  *home = h;
  return true;
}

PlannedStart LaunchState::current(const PlannedStart& ps) const {
  if (resizes_[ps.model] == 0) return ps;
  return PlannedStart{ps.t, ps.model, range_mask(home_[ps.model], dep_[ps.model]),
                      table_latency(ps.model, plan_->batch[ps.model], dep_[ps.model])};
}

bool LaunchState::temporal_pick(int64_t t, Pick* out) const {
  if (t >= D_ || used_ != 0) return false;
  const int64_t r = t % cycle_;
  int i = -1;
  for (int j = 0; j < n_; ++j)
    if (r >= slice_off_[j] && r < slice_off_[j] + slice_len_[j]) i = j;
  if (i < 0 || queue_[i].empty()) return false;
  const int64_t left = slice_off_[i] + slice_len_[i] - r;
  const int total = prm_->total_slots;
  int bb = -1;
  int64_t bL = 0;
  for (int b : kGrid) {
    if (b > models_[i].max_batch || b > (int)queue_[i].size()) continue;
    const int64_t L = table_latency(i, b, total);
    if (L <= 0 || L > left) continue;
    bb = b;
    bL = L;
  }
  if (bb < 0) return false;
  *out = Pick{i, range_mask(0, total), bb, bL};
  return true;
}

int64_t LaunchState::table_latency(int i, int b, int slots) const {
  const dstack_sched_model& m = models_[i];
  int row = -1;
  for (int q = 0; q < m.n_batches; ++q)
    if (m.batches[q] == b) row = q;
  if (row < 0) return -1;
  int64_t L = -1;
  for (int q = 0; q < m.n_slots; ++q)
    if (m.slots[q] <= slots && m.latency_us[row][q] > 0) L = m.latency_us[row][q];
  return L;
}

bool LaunchState::fod_pick(int64_t t, Pick* out) const {
  if (t >= D_) return false;  // nothing starts once the trace has ended
  std::vector<int> cands;
  for (int i = 0; i < n_; ++i)
    if (!running_[i] && !queue_[i].empty() && avail_[i]) cands.push_back(i);
  const int64_t cur = t / T_;
  auto recent = [&](int i) {
    int64_t r = 0;
    for (auto it = runs_[i].lower_bound(cur - sim_->sessions_window + 1); it != runs_[i].end() && it->first <= cur;
         ++it)
      r += it->second;
    return r;
  };
  std::stable_sort(cands.begin(), cands.end(), [&](int a, int b) {
    if (sim_->policy == 1) {  // least runtime first
      if (plan_->latency_us[a] != plan_->latency_us[b]) return plan_->latency_us[a] < plan_->latency_us[b];
      return a < b;
    }
    if (sim_->policy == 2) {  // smallest GPU% demand first
      if (plan_->deployed_slots[a] != plan_->deployed_slots[b])
        return plan_->deployed_slots[a] < plan_->deployed_slots[b];
      if (busy_[a] != busy_[b]) return busy_[a] < busy_[b];
      return a < b;
    }
    int64_t ra = recent(a), rb = recent(b);
    if (ra != rb) return ra < rb;
    if (busy_[a] != busy_[b]) return busy_[a] < busy_[b];
    return a < b;
  });
  const int total = prm_->total_slots;
  for (int i : cands) {
    const int s = dep_[i];
    uint64_t mask = 0;
    if (prm_->placement == 1) {
      mask = range_mask(home_[i], s);
      if (used_ & mask) continue;
    } else {
      int got = 0;
      for (int sid = 0; sid < total && got < s; ++sid)
        if (!((used_ >> sid) & 1)) {
          mask |= 1ULL << sid;
          ++got;
        }
      if (got < s) continue;
    }
    // -1: no planned start constrains it; a planned start at this very
    // instant counts (same-instant planned starts are processed after
    // completions)
    int64_t gap = -1;
    for (const PlannedStart& p0 : pstarts_) {
      const PlannedStart ps = current(p0);
      if (ps.t >= t && ((ps.mask & mask) || ps.model == i)) {
        gap = ps.t - t;
        break;
      }
    }
    int bb = -1;
    int64_t bL = 0;
    for (int b : kGrid) {
      if (b > models_[i].max_batch || b > (int)queue_[i].size()) continue;
      const int64_t L = table_latency(i, b, s);
      if (L <= 0 || (gap >= 0 && L > gap)) continue;
      bb = b;
      bL = L;
    }
    if (bb < 0) continue;
    *out = Pick{i, mask, bb, bL};
    return true;
  }
  return false;
}

std::vector<int64_t> LaunchState::start(int64_t t, int i, uint64_t mask, int64_t charged_us, int b) {
  std::vector<int64_t> reqs;
  for (int k = 0; k < b; ++k) {
    reqs.push_back(queue_[i].front());
    queue_[i].pop_front();
  }
  if (sim_->policy == 0 && sim_->resize_violations > 0)
    for (int64_t a : reqs)
      if (a >= changed_at_[i] && 2 * (t - a) > models_[i].slo_us) viol_[i] += 1;
  running_[i] = 1;
  run_mask_[i] = mask;
  used_ |= mask;
  runs_[i][t / T_] += 1;
  busy_[i] += charged_us;
  return reqs;
}

void LaunchState::finish(int i) {
  running_[i] = 0;
  used_ &= ~run_mask_[i];
}

dstack_status simulate(const dstack_sched_model* models, int n, const dstack_sched_params* prm,
                       const dstack_sim_params* sim, dstack_run_out* out) {
  DS_CHECK(sim && out && prm, DSTACK_E_INVALID, "simulate: null pointer");
  DS_CHECK(n >= 1 && n <= DSTACK_MAX_MODELS, DSTACK_E_INVALID, "simulate: bad model count");
  DS_CHECK(check_trace(n, sim), DSTACK_E_INVALID,
           "simulate: bad trace (duration > 0, window >= 1, policy 0..3, arrivals sorted inside [0, duration))");
  DS_CHECK(sim->resize_violations == 0 || (sim->policy == 0 && prm->placement == 1), DSTACK_E_INVALID,
           "simulate: GPU% changes on SLO violations need the D-STACK policy with home placement");
  std::vector<dstack_schedule_out> plan_box(1);
  dstack_schedule_out* plan = &plan_box[0];
  dstack_status st = schedule(models, n, prm, plan);
  if (st != DSTACK_OK && st != DSTACK_E_INFEASIBLE) return st;
  const int64_t D = sim->duration_us;
  const int total = prm->total_slots;
  LaunchState ls(models, n, prm, sim, plan);

  std::priority_queue<Event, std::vector<Event>, std::greater<Event>> ev;
  int64_t seq = 0;
  for (const PlannedStart& ps : ls.planned()) ev.push(Event{ps.t, 1, ps.model, seq++, ps.mask, ps.dur, {}});
  for (const PlannedStart& ps : ls.slice_starts()) ev.push(Event{ps.t, 1, ps.model, seq++, ps.mask, 0, {}});
  for (int i = 0; i < n; ++i)
    for (int k = 0; k < sim->n_arrivals[i]; ++k) ev.push(Event{sim->arrivals_us[i][k], 2, i, seq++, 0, 0, {}});

  std::vector<int64_t> served(n, 0), late(n, 0), pruns(n, 0), fruns(n, 0), skips(n, 0), busy(n, 0);
  std::vector<std::vector<int64_t>> lats(n);
  int64_t slot_us = 0, last_end = 0;
  uint64_t h = kFnvOffset;

  auto launch = [&](int64_t t, int i, uint64_t mask, int64_t dur, int b, int kind) {
    Event c{t + dur, 0, i, seq++, mask, dur, ls.start(t, i, mask, dur, b)};
    ev.push(std::move(c));
    busy[i] += dur;
    slot_us += (int64_t)__builtin_popcountll(mask) * (std::min(t + dur, D) - t);  // slot-time inside [0, D)
    last_end = std::max(last_end, t + dur);
    for (int64_t v : {t, (int64_t)i, (int64_t)b, (int64_t)mask, dur, (int64_t)kind}) h = fnv_mix(h, v);
    (kind == 0 ? pruns : fruns)[i] += 1;
  };
  auto fod_pass = [&](int64_t t) {
    LaunchState::Pick pk;
    if (ls.temporal()) {
      if (ls.temporal_pick(t, &pk)) launch(t, pk.model, pk.mask, pk.latency, pk.batch, 0);
    } else if ((sim->fod || sim->policy != 0) && ls.fod_pick(t, &pk)) {
      launch(t, pk.model, pk.mask, pk.latency, pk.batch, 1);
    }
  };

  while (!ev.empty()) {
    Event e = ev.top();
    ev.pop();
    const int i = e.model;
    if (e.kind == 0) {
      ls.finish(i);
      int64_t job_late = 0;
      for (int64_t a : e.reqs) {
        served[i] += 1;
        lats[i].push_back(e.t - a);
        if (e.t - a > models[i].slo_us) job_late += 1;
      }
      late[i] += job_late;
      ls.note_late(e.t, i, ls.late_at_end(i, e.t - e.dur, e.t, e.reqs));
      fod_pass(e.t);
    } else if (e.kind == 1 && ls.temporal()) {
      fod_pass(e.t);
    } else if (e.kind == 1) {
      // a planned start (its model may have changed size since the plan)
      const PlannedStart ps = ls.current(PlannedStart{e.t, i, e.mask, e.dur});
      if (ls.queued(i) && !ls.running(i) && ls.free(ps.mask))
        launch(e.t, i, ps.mask, ps.dur, std::min<int>(ls.plan_batch(i), (int)ls.queued(i)), 0);
      else
        skips[i] += 1;
    } else {
      ls.arrive(i, e.t);
      fod_pass(e.t);
    }
  }

  std::memset(out, 0, sizeof(*out));
  out->n_models = n;
  for (int i = 0; i < n; ++i) {
    dstack_model_stats& s = out->models[i];
    s.served = served[i];
    s.unserved = (int64_t)ls.queued(i);
    s.violations = late[i] + s.unserved;
    s.planned_runs = pruns[i];
    s.fod_runs = fruns[i];
    s.busy_us = busy[i];
    s.p50_us = nearest_rank(lats[i], 50);
    s.p99_us = nearest_rank(lats[i], 99);
    s.plan_skips = skips[i];
    s.resizes = ls.resizes(i);
    s.final_slots = ls.temporal() ? total : ls.deployed(i);
  }
  out->utilisation_ppm = (int64_t)((unsigned __int128)slot_us * 1000000 / ((unsigned __int128)total * (uint64_t)D));
  out->job_hash = h;
  out->last_end_us = last_end;
  return DSTACK_OK;
}

// The ideal spatio-temporal schedule of Sec. 6.2 (Eqs. maximization and
// constraints): slotted, kernel granularity, preemptive; every slot runs the
// subset of the models' current kernels with the largest summed share that
// fits, found by exhaustive search (2^n subsets, n <= 8).
dstack_status simulate_ideal(const dstack_ideal_model* models, int n, int64_t horizon, int64_t slot, int total,
                             dstack_ideal_out* out) {
  DS_CHECK(models && out, DSTACK_E_INVALID, "simulate_ideal: null pointer");
  DS_CHECK(n >= 1 && n <= 8 && horizon >= 1 && slot >= 1 && total >= 1 && total <= 64, DSTACK_E_INVALID,
           "simulate_ideal: 1..8 models, horizon >= 1, slot >= 1, total 1..64");
  for (int i = 0; i < n; ++i) {
    const dstack_ideal_model& m = models[i];
    DS_CHECK(m.n_kernels >= 1 && m.slots && m.dur_us && m.batch >= 1 && m.slo_us >= 1, DSTACK_E_INVALID,
             "simulate_ideal: a model needs kernels, batch >= 1 and slo >= 1");
    for (int k = 0; k < m.n_kernels; ++k)
      DS_CHECK(m.slots[k] >= 1 && m.slots[k] <= total && m.dur_us[k] >= 1, DSTACK_E_INVALID,
               "simulate_ideal: kernel shares 1..total and durations >= 1 us");
  }
  std::vector<int> k(n, 0);
  std::vector<int64_t> rem(n), deadline(n), items(n, 0), fwd(n, 0), late(n, 0), busy(n, 0);
  for (int i = 0; i < n; ++i) {
    rem[i] = models[i].dur_us[0];
    deadline[i] = models[i].slo_us;
  }
  int64_t used_sum = 0, n_slots = 0;
  uint64_t h = kFnvOffset;
  std::vector<int> order(n);
  for (int64_t t = 0; t < horizon; t += slot) {
    for (int i = 0; i < n; ++i) order[i] = i;
    std::stable_sort(order.begin(), order.end(), [&](int a, int b) {
      if (deadline[a] != deadline[b]) return deadline[a] < deadline[b];
      return a < b;
    });
    int best = 0, best_sum = -1;
    unsigned best_bits = 0;
    for (int sub = 0; sub < (1 << n); ++sub) {
      int s = 0;
      for (int i = 0; i < n; ++i)
        if ((sub >> i) & 1) s += models[i].slots[k[i]];
      if (s > total) continue;
      unsigned bits = 0;
      for (int i : order) bits = (bits << 1) | ((sub >> i) & 1);
      if (s > best_sum || (s == best_sum && bits > best_bits)) {
        best_sum = s;
        best_bits = bits;
        best = sub;
      }
    }
    used_sum += best_sum;
    n_slots += 1;
    h = fnv_mix(h, t);
    h = fnv_mix(h, best);
    const int64_t end = t + slot;
    for (int i = 0; i < n; ++i) {
      if (!((best >> i) & 1)) continue;
      busy[i] += (int64_t)models[i].slots[k[i]] * slot;
      rem[i] -= slot;
      if (rem[i] <= 0) {
        k[i] += 1;
        if (k[i] == models[i].n_kernels) {
          fwd[i] += 1;
          items[i] += models[i].batch;
          if (end > deadline[i]) late[i] += 1;
          k[i] = 0;
          deadline[i] = end + models[i].slo_us;
        }
        rem[i] = models[i].dur_us[k[i]];
      }
    }
  }
  std::memset(out, 0, sizeof(*out));
  out->n_models = n;
  for (int i = 0; i < n; ++i) {
    out->items[i] = items[i];
    out->forwards[i] = fwd[i];
    out->late[i] = late[i];
    out->busy_slot_us[i] = busy[i];
  }
  out->utilisation_ppm = used_sum * 1000000 / ((int64_t)total * std::max<int64_t>(n_slots, 1));
  out->hash = h;
  return DSTACK_OK;
}

}  // namespace dstack
