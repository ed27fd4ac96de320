// Host-side decisions of D-STACK: knee, SLO-constrained batch choice and the
// spatio-temporal session plan.  Pure integer arithmetic on a measured
// timing table L[b][s] (microseconds), so the result is a deterministic
// function of the table.
//
//  * Efficacy (Sec. 5, Eqs. efficiency / efficiencySquareLatency):
//    eta = b / (L^2 * s); compared exactly in 128-bit integers.
//  * Batch/GPU% optimisation (Sec. 5.1, Eqs. max_batch_size, meet_slo,
//    meet_half_slo) as an exhaustive search over the measured grid (the
//    paper fits f_L and calls a continuous solver; the grid is exact here).
//  * Session plan (Sec. 6.1, 6.1.1): EDF over per-SLO windows, consecutive
//    runs pushed apart (even runs early, odd runs late), no over-subscription,
//    below-knee fallback, no preemption.
//  * Placement: lowest free slot ids per job, or fixed home ranges (one
//    contiguous range of the deployed size per model, the launcher's one
//    CU-masked stream per model); a home job needs its whole range free.
#include <algorithm>
#include <cstring>
#include <vector>

#include "sched.hpp"

namespace dstack {

typedef unsigned __int128 u128;

bool eta_greater(int64_t b1, int64_t L1, int64_t s1, int64_t b2, int64_t L2, int64_t s2) {
  return (u128)b1 * (u128)L2 * (u128)L2 * (u128)s2 > (u128)b2 * (u128)L1 * (u128)L1 * (u128)s1;
}

int knee_index(int b, const int64_t* lat, const int* slots, int n) {
  int best = -1;
  for (int i = 0; i < n; ++i) {
    if (lat[i] <= 0) continue;
    if (best < 0) {
      best = i;
      continue;
    }
    // strictly better efficacy wins; equal efficacy keeps the fewer slots
    if (eta_greater(b, lat[i], slots[i], b, lat[best], slots[best]) ||
        (!eta_greater(b, lat[best], slots[best], b, lat[i], slots[i]) && slots[i] < slots[best]))
      best = i;
  }
  return best;
}

int knee_search(int b, const std::vector<int>& cand, int start, const std::function<int64_t(int)>& latency,
                std::vector<std::pair<int, int64_t>>* probes) {
  const int n = (int)cand.size();
  std::vector<int64_t> seen(n, 0);
  auto L = [&](int i) {
    if (!seen[i]) {
      seen[i] = latency(cand[i]);
      probes->push_back({cand[i], seen[i]});
    }
    return seen[i];
  };
  int lo = 0, hi = n - 1, mid = 0;
  for (int i = 0; i < n; ++i)
    if (cand[i] <= start) mid = i;
  while (lo < hi) {
    mid = std::min(std::max(mid, lo), hi - 1);
    const int64_t a = L(mid), c = L(mid + 1);
    if (eta_greater(b, c, cand[mid + 1], b, a, cand[mid]))
      lo = mid + 1;  // the next candidate still raises the efficacy
    else
      hi = mid;
    mid = lo + (hi - lo) / 2;
  }
  // confirmation against the grid neighbours k-2, k-1, k+1, k+2: latency
  // falls in steps, so the bisection can stop on a local maximum of eta
  auto better = [&](int j, int i) {
    const int64_t lj = L(j), li = L(i);
    return eta_greater(b, lj, cand[j], b, li, cand[i]) ||
           (!eta_greater(b, li, cand[i], b, lj, cand[j]) && cand[j] < cand[i]);
  };
  int k = lo;
  for (;;) {
    int best = k;
    for (int j : {k - 2, k - 1, k + 1, k + 2})
      if (j >= 0 && j < n && better(j, best)) best = j;
    if (best == k) return k;
    k = best;
  }
}

namespace {

const int kBatchGrid[] = {1, 2, 4, 8, 16, 32};

int64_t assembly_time(int b, int rate) {
  if (rate > 0) return ((int64_t)b * 1000000 + rate - 1) / rate;
  return 482LL * b;
}

struct Row {
  std::vector<int> s;       // ascending swept slot counts
  std::vector<int64_t> L;   // latency at each
  int64_t at(int slots) const {  // measurement at the largest swept count <= slots
    int64_t r = -1;
    for (size_t i = 0; i < s.size(); ++i)
      if (s[i] <= slots) r = L[i];
    return r;
  }
};

struct Placed {
  int64_t start, end;
  int slots;
  int job;
  uint64_t mask;  // home placement: the range it occupies
};

// Largest total slots of placed jobs at any instant in [t0, t1).  The load is
// piecewise constant and only rises at job starts, so it is enough to look
// at t0 and at every start inside the interval.
int peak_load(const std::vector<Placed>& placed, int64_t t0, int64_t t1) {
  int peak = 0;
  auto load_at = [&](int64_t t) {
    int l = 0;
    for (const Placed& p : placed)
      if (p.start <= t && t < p.end) l += p.slots;
    return l;
  };
  peak = load_at(t0);
  for (const Placed& p : placed)
    if (p.start > t0 && p.start < t1) peak = std::max(peak, load_at(p.start));
  return peak;
}

// home placement: does a placed job overlapping [t0, t1) use a slot of mask?
bool conflicts(const std::vector<Placed>& placed, int64_t t0, int64_t t1, uint64_t mask) {
  for (const Placed& p : placed)
    if (p.start < t1 && t0 < p.end && (p.mask & mask)) return true;
  return false;
}

// home_mask == 0: feasible when the summed slots stay within the total;
// otherwise when no overlapping job meets the home range
bool find_start(const std::vector<Placed>& placed, int64_t ws, int64_t we, int64_t L, int s, bool latest, int total,
                uint64_t home_mask, int64_t* out) {
  if (L > we - ws) return false;
  std::vector<int64_t> cand;
  cand.push_back(ws);
  cand.push_back(we - L);
  for (const Placed& p : placed) {
    cand.push_back(p.end);
    cand.push_back(p.start - L);
  }
  std::vector<int64_t> ok;
  for (int64_t c : cand)
    if (c >= ws && c <= we - L) ok.push_back(c);
  std::sort(ok.begin(), ok.end());
  ok.erase(std::unique(ok.begin(), ok.end()), ok.end());
  if (latest) std::reverse(ok.begin(), ok.end());
  for (int64_t t : ok) {
    const bool fits = home_mask ? !conflicts(placed, t, t + L, home_mask) : peak_load(placed, t, t + L) + s <= total;
    if (fits) {
      *out = t;
      return true;
    }
  }
  return false;
}

}  // namespace

void home_offsets(const int* sizes, int n, int total, int* offs) {
  std::vector<int> order(n);
  for (int i = 0; i < n; ++i) order[i] = i;
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return sizes[a] > sizes[b]; });
  std::vector<std::pair<int, int>> placed;  // (offset, size)
  for (int i : order) {
    int best = -1, best_ov = 0;
    for (int o = 0; o + sizes[i] <= total; ++o) {
      int ov = 0;
      for (auto& p : placed) ov += std::max(0, std::min(o + sizes[i], p.first + p.second) - std::max(o, p.first));
      if (best < 0 || ov < best_ov) {
        best = o;
        best_ov = ov;
      }
    }
    offs[i] = best;
    placed.push_back({best, sizes[i]});
  }
}

uint64_t range_mask(int offset, int size) {
  return (size >= 64 ? ~0ULL : ((1ULL << size) - 1)) << offset;
}

dstack_status schedule(const dstack_sched_model* models, int n, const dstack_sched_params* prm,
                       dstack_schedule_out* out) {
  DS_CHECK(models && prm && out, DSTACK_E_INVALID, "schedule: null pointer");
  DS_CHECK(n >= 1 && n <= DSTACK_MAX_MODELS, DSTACK_E_INVALID, "schedule: 1..16 models");
  DS_CHECK(prm->period_us > 0 && prm->total_slots >= 1 && prm->total_slots <= 64 && prm->overprov_slots >= 0 &&
               (prm->placement == 0 || prm->placement == 1),
           DSTACK_E_INVALID, "schedule: bad params");
  std::memset(out, 0, sizeof(*out));
  out->n_models = n;
  const int total = prm->total_slots;
  bool any_infeasible = false;

  std::vector<Row> rows(n);
  std::vector<int> knee(n), deployed(n);
  std::vector<int64_t> slo(n);
  for (int i = 0; i < n; ++i) {
    const dstack_sched_model& m = models[i];
    DS_CHECK(m.slo_us > 0 && m.max_batch >= 1 && m.n_batches >= 1 && m.n_batches <= DSTACK_MAX_BATCHES &&
                 m.n_slots >= 1 && m.n_slots <= DSTACK_MAX_SWEEP && m.rate_per_s >= 0,
             DSTACK_E_INVALID, "schedule: bad model entry");
    for (int j = 1; j < m.n_slots; ++j)
      DS_CHECK(m.slots[j] > m.slots[j - 1], DSTACK_E_INVALID, "schedule: slot counts must ascend");
    DS_CHECK(m.slots[0] >= 1 && m.slots[m.n_slots - 1] <= total, DSTACK_E_INVALID, "schedule: slot count out of range");
    slo[i] = m.slo_us;
    // exhaustive search over the measured (b, s) grid
    int bb = -1, bs = -1;
    int64_t bL = 0;
    for (int g : kBatchGrid) {
      if (g > m.max_batch) continue;
      int r = -1;
      for (int q = 0; q < m.n_batches; ++q)
        if (m.batches[q] == g) r = q;
      if (r < 0) continue;
      const int64_t C = assembly_time(g, m.rate_per_s);
      for (int q = 0; q < m.n_slots; ++q) {
        const int64_t L = m.latency_us[r][q];
        if (L <= 0) continue;
        if (L + C > m.slo_us || L > m.slo_us / 2) continue;
        const int s = m.slots[q];
        bool take;
        if (bb < 0)
          take = true;
        else if (eta_greater(g, L, s, bb, bL, bs))
          take = true;
        else if (eta_greater(bb, bL, bs, g, L, s))
          take = false;
        else
          take = s < bs || (s == bs && g > bb);
        if (take) {
          bb = g;
          bs = s;
          bL = L;
        }
      }
    }
    int row_q = -1;
    if (bb >= 0) {
      out->feasible[i] = 1;
    } else {
      any_infeasible = true;
      // b = 1 if measured, else the smallest measured batch; its lowest latency
      int pick = -1;
      for (int q = 0; q < m.n_batches; ++q)
        if (pick < 0 || (m.batches[q] == 1) || (m.batches[pick] != 1 && m.batches[q] < m.batches[pick])) pick = q;
      bb = m.batches[pick];
      for (int q = 0; q < m.n_slots; ++q) {
        const int64_t L = m.latency_us[pick][q];
        if (L <= 0) continue;
        if (bs < 0 || L < bL) {
          bs = m.slots[q];
          bL = L;
        }
      }
      DS_CHECK(bs >= 0, DSTACK_E_INVALID, "schedule: a model has no measured latency");
    }
    for (int q = 0; q < m.n_batches; ++q)
      if (m.batches[q] == bb) row_q = q;
    for (int q = 0; q < m.n_slots; ++q)
      if (m.latency_us[row_q][q] > 0) {
        rows[i].s.push_back(m.slots[q]);
        rows[i].L.push_back(m.latency_us[row_q][q]);
      }
    knee[i] = bs;
    deployed[i] = std::min(total, bs + prm->overprov_slots);
    out->batch[i] = bb;
    out->knee_slots[i] = bs;
    out->deployed_slots[i] = deployed[i];
    out->latency_us[i] = bL;
  }

  const bool home = prm->placement == 1;
  std::vector<uint64_t> hmask(n, 0);
  if (home) {
    home_offsets(deployed.data(), n, total, out->home_offset);
    for (int i = 0; i < n; ++i) hmask[i] = range_mask(out->home_offset[i], deployed[i]);
  }

  // jobs in EDF order (deadline, SLO, model, k)
  struct J {
    int model, k;
    int64_t ws, we;
  };
  std::vector<J> jobs;
  const int64_t T = prm->period_us;
  for (int i = 0; i < n; ++i) {
    int64_t r = (T + slo[i] - 1) / slo[i];
    for (int64_t k = 0; k < r; ++k) jobs.push_back(J{i, (int)k, k * slo[i], std::min((k + 1) * slo[i], T)});
  }
  DS_CHECK(jobs.size() <= DSTACK_MAX_JOBS, DSTACK_E_INVALID, "schedule: more than 512 jobs per period");
  std::stable_sort(jobs.begin(), jobs.end(), [&](const J& a, const J& b) {
    if (a.we != b.we) return a.we < b.we;
    if (slo[a.model] != slo[b.model]) return slo[a.model] < slo[b.model];
    if (a.model != b.model) return a.model < b.model;
    return a.k < b.k;
  });

  std::vector<Placed> placed;
  out->n_jobs = (int)jobs.size();
  for (size_t o = 0; o < jobs.size(); ++o) {
    const J& j = jobs[o];
    dstack_job& dj = out->jobs[o];
    dj.model = j.model;
    dj.k = j.k;
    dj.release_us = j.ws;
    dj.deadline_us = j.we;
    // deployed slots, then the knee, then every smaller swept count (home
    // placement: the home range only)
    std::vector<int> opts{deployed[j.model]};
    const Row& row = rows[j.model];
    if (!home) {
      if (knee[j.model] != deployed[j.model]) opts.push_back(knee[j.model]);
      for (int q = (int)row.s.size() - 1; q >= 0; --q)
        if (row.s[q] < knee[j.model]) opts.push_back(row.s[q]);
    }
    bool done = false;
    for (int s : opts) {
      int64_t L = row.at(s);
      if (L <= 0) continue;
      int64_t t;
      if (find_start(placed, j.ws, j.we, L, s, (j.k & 1) != 0, total, hmask[j.model], &t)) {
        dj.start_us = t;
        dj.duration_us = L;
        dj.slots = s;
        dj.slot_mask = hmask[j.model];
        placed.push_back(Placed{t, t + L, s, (int)o, hmask[j.model]});
        done = true;
        break;
      }
    }
    if (!done) {
      dj.start_us = j.ws;
      dj.duration_us = 0;
      dj.slots = 0;
      dj.missed = 1;
      any_infeasible = true;
    }
  }

  // slot ids: in (start, placement order), lowest free ids at the start
  std::vector<Placed> order = home ? std::vector<Placed>() : placed;
  std::stable_sort(order.begin(), order.end(), [](const Placed& a, const Placed& b) {
    if (a.start != b.start) return a.start < b.start;
    return a.job < b.job;
  });
  std::vector<std::pair<int64_t, uint64_t>> busy;  // (end, mask)
  for (const Placed& p : order) {
    uint64_t used = 0;
    for (auto& e : busy)
      if (e.first > p.start) used |= e.second;
    uint64_t mask = 0;
    int need = p.slots;
    for (int sid = 0; sid < total && need > 0; ++sid)
      if (!((used >> sid) & 1)) {
        mask |= 1ULL << sid;
        --need;
      }
    DS_CHECK(need == 0, DSTACK_E_STATE, "schedule: slot assignment failed");
    out->jobs[p.job].slot_mask = mask;
    busy.push_back({p.end, mask});
  }

  u128 num = 0;
  for (const Placed& p : placed) num += (u128)p.slots * (u128)(p.end - p.start);
  out->utilisation_ppm = (int64_t)(num * 1000000 / ((u128)total * (u128)T));
  if (any_infeasible) return fail(DSTACK_E_INFEASIBLE, "schedule: infeasible model or missed job (plan filled)");
  return DSTACK_OK;
}

}  // namespace dstack
