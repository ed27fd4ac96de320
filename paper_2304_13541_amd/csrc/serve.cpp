// Live launcher: the session plan and the FOD fill of Sec. 6.1.2 driving
// real batches on CU-masked streams.  Model i runs on a partition over its
// home range (the plan's home placement); models whose ranges are identical
// share one (a job needs its whole range free, so their jobs never overlap),
// and at most four masked streams exist at once.  A slot the sharing leaves
// free holds a standby: the stream of the next larger range of a model that
// has started to miss its SLO, created ahead on a helper thread, so that its
// GPU% change (Sec. 3.5's active-standby pair) takes effect at once.  The
// host thread follows the request trace on its monotonic clock,
// launches planned and FOD jobs through dstack_infer, and polls each job's
// end event.  The decisions are those of the virtual-clock simulation (the
// same LaunchState, fed with table latencies); only the completion times and
// GPU durations are measured.  Every trigger (a completion seen, a planned
// or slice start due, an arrival admitted) is logged with the clock value
// its decision used, so that the decisions can be replayed off the GPU.
// The temporal-sharing baseline (policy 3) runs the same loop with slice
// starts in place of planned starts, every model on one whole-GPU partition.
#include <hip/hip_runtime.h>

#include <chrono>
#include <cmath>
#include <atomic>
#include <condition_variable>
#include <cstring>
#include <deque>
#include <functional>
#include <memory>
#include <future>
#include <mutex>
#include <string>
#include <thread>
#include <utility>
#include <vector>

#include "launcher.hpp"

namespace dstack {

namespace {

int64_t host_us() {
  return std::chrono::duration_cast<std::chrono::microseconds>(std::chrono::steady_clock::now().time_since_epoch())
      .count();
}

constexpr int kMaxServeModels = 4;
static_assert(kMaxServeModels <= kLauncherWsCount, "one launcher workspace per model");
constexpr int kResizeAhead = 5;  // GPU% changes per model whose graphs the warm-up captures
constexpr int64_t kDrainLimitUs = 60LL * 1000 * 1000;  // a job still running this long after the trace: error
const int kGrid[] = {1, 2, 4, 8, 16, 32};

struct Running {
  bool on = false;
  int64_t start = 0, table_us = 0;
  uint64_t mask = 0;
  int batch = 0, kind = 0;
  std::vector<int64_t> reqs;
};

// A GPU% change's new partition, created on a helper thread so that the
// launcher keeps serving the other models meanwhile.  The error text is
// carried back because dstack_last_error() is per thread.
struct NewPartition {
  dstack_status first = DSTACK_OK;
  dstack_partition second = nullptr;
  std::string err;
};

// Partition creations and destructions run on one helper thread in the
// order they are submitted, so that the launcher thread never waits for a
// stream to be made or torn down (a stream's destruction can take
// milliseconds), and a creation submitted after a destruction runs after it
// (the live count then never passes the library's limit).  Queued work is
// finished before the thread ends.
class PartitionWorker {
 public:
  explicit PartitionWorker(int dev) : dev_(dev), th_([this] { loop(); }) {}
  ~PartitionWorker() {
    {
      std::lock_guard<std::mutex> g(mu_);
      stop_ = true;
    }
    cv_.notify_all();
    th_.join();
  }
  std::future<NewPartition> create(int off, int cnt) {
    auto task = std::make_shared<std::packaged_task<NewPartition()>>([this, off, cnt] {
      NewPartition np;
      if (dev_err_ != hipSuccess) {
        np.first = DSTACK_E_HIP;
        np.err = std::string("serve: hipSetDevice: ") + hipGetErrorString(dev_err_);
      } else {
        np.first = dstack_partition_create_at(off, cnt, &np.second);
        if (np.first != DSTACK_OK) np.err = dstack_last_error();
      }
      return np;
    });
    std::future<NewPartition> f = task->get_future();
    creates_.fetch_add(1);
    submit([this, task] {
      (*task)();
      creates_.fetch_sub(1);  // after the new partition counts as live
    });
    return f;
  }
  void destroy(dstack_partition p) {
    destroys_.fetch_add(1);
    submit([this, p] {
      destroys_.fetch_sub(1);  // before it stops counting as live
      dstack_partition_destroy(p);
    });
  }
  // submitted and not finished yet
  int creates() const { return creates_.load(); }
  int destroys() const { return destroys_.load(); }

 private:
  void submit(std::function<void()> f) {
    {
      std::lock_guard<std::mutex> g(mu_);
      q_.emplace_back(std::move(f));
    }
    cv_.notify_one();
  }
  void loop() {
    dev_err_ = hipSetDevice(dev_);  // a new thread starts on device 0
    for (;;) {
      std::function<void()> f;
      {
        std::unique_lock<std::mutex> g(mu_);
        cv_.wait(g, [this] { return stop_ || !q_.empty(); });
        if (q_.empty()) return;  // stop_ and nothing left
        f = std::move(q_.front());
        q_.pop_front();
      }
      f();
    }
  }
  int dev_;
  hipError_t dev_err_ = hipSuccess;
  std::mutex mu_;
  std::condition_variable cv_;
  std::deque<std::function<void()>> q_;
  bool stop_ = false;
  std::atomic<int> creates_{0}, destroys_{0};
  std::thread th_;  // last: starts after the members it uses
};

// A live partition and the models whose current range it covers.
struct PoolEntry {
  int off = 0, n = 0, users = 0;
  dstack_partition p = nullptr;
  hipStream_t s = nullptr;
};

struct Resources {
  std::unique_ptr<PartitionWorker> worker;           // made after the first partitions
  std::vector<PoolEntry> pool;                      // p == nullptr: a free entry
  std::vector<std::future<NewPartition>> pending;  // per model; valid() while a stream of its next range is created
  std::vector<dstack_partition> made;              // per model: that stream, created and not used yet
  std::vector<int> made_off, made_n;               // the range pending[i] / made[i] covers
  std::vector<hipEvent_t> ev0, ev1;
  bool drained = true;  // false: a job may still run, keep the partitions that ran jobs
  ~Resources() {
    worker.reset();  // finishes the queued creations and destructions
    for (size_t i = 0; i < pending.size(); ++i)
      if (pending[i].valid()) {  // an early return: the creation is done
        NewPartition np = pending[i].get();
        if (np.first == DSTACK_OK) made[i] = np.second;
      }
    for (hipEvent_t e : ev0)
      if (e) (void)hipEventDestroy(e);
    for (hipEvent_t e : ev1)
      if (e) (void)hipEventDestroy(e);
    for (dstack_partition p : made)  // never ran a job
      if (p) dstack_partition_destroy(p);
    if (drained)
      for (const PoolEntry& e : pool)
        if (e.p) dstack_partition_destroy(e.p);
  }
};

}  // namespace

dstack_status serve(const dstack_model* models, int n, const void* const* d_in, void* const* d_out,
                    const dstack_sched_model* tables, const dstack_sched_params* prm, const dstack_sim_params* sim,
                    dstack_run_out* out, dstack_job_record* log, int log_capacity, int* n_log,
                    dstack_serve_event* events, int event_capacity, int* n_events) {
  DS_CHECK(models && d_in && d_out && tables && prm && sim && out, DSTACK_E_INVALID, "serve: null pointer");
  DS_CHECK(n >= 1 && n <= DSTACK_MAX_MODELS, DSTACK_E_INVALID, "serve: bad model count");
  DS_CHECK(n <= kMaxServeModels, DSTACK_E_UNSUPPORTED, "serve: at most 4 models (at most one CU-masked stream each)");
  DS_CHECK(log_capacity >= 0 && (log || log_capacity == 0), DSTACK_E_INVALID, "serve: bad log buffer");
  DS_CHECK(event_capacity >= 0 && (events || event_capacity == 0), DSTACK_E_INVALID, "serve: bad event buffer");
  DS_CHECK(check_trace(n, sim), DSTACK_E_INVALID, "serve: bad trace (see dstack_simulate)");
  DS_CHECK(sim->policy == 0 || sim->policy == 3, DSTACK_E_INVALID,
           "serve: runs the D-STACK policy (0) or temporal sharing (3)");
  const bool temporal = sim->policy == 3;
  DS_CHECK(temporal || prm->placement == 1, DSTACK_E_INVALID, "serve: D-STACK needs placement 1 (home ranges)");
  DS_CHECK(!temporal || sim->resize_violations == 0, DSTACK_E_INVALID,
           "serve: GPU% changes on SLO violations are a D-STACK feature (policy 0)");
  DS_CHECK(prm->total_slots >= 1 && prm->total_slots <= DSTACK_TOTAL_SLOTS, DSTACK_E_INVALID,
           "serve: total_slots must be in 1..32 (one GPU)");
  for (int i = 0; i < n; ++i) {
    DS_CHECK(models[i] && d_in[i] && d_out[i], DSTACK_E_INVALID, "serve: null model or buffer");
    dstack_model_info q;
    dstack_status s = dstack_model_query(models[i], &q);
    if (s != DSTACK_OK) return s;
    DS_CHECK(tables[i].max_batch >= 1 && tables[i].max_batch <= q.max_batch, DSTACK_E_INVALID,
             "serve: table max_batch above the model's");
  }
  std::vector<dstack_schedule_out> plan_box(1);
  dstack_schedule_out* plan = &plan_box[0];
  dstack_status st = schedule(tables, n, prm, plan);
  if (st != DSTACK_OK && st != DSTACK_E_INFEASIBLE) return st;

  // D-STACK: model i runs on a partition over its home range, shared with
  // the models of the same range.  Temporal sharing: one partition of all
  // the slots, which every model's jobs use in turn.
  Resources res;
  res.pending.resize(n);
  res.made.assign(n, nullptr);
  res.made_off.assign(n, -1);
  res.made_n.assign(n, 0);
  res.ev0.assign(n, nullptr);
  res.ev1.assign(n, nullptr);
  std::vector<int> cur(n, -1);  // model i's pool entry (-1 while it waits for a new one)
  std::vector<dstack_partition> part(n);
  std::vector<hipStream_t> stream(n);
  auto find_entry = [&](int off, int cnt) {
    for (size_t k = 0; k < res.pool.size(); ++k)
      if (res.pool[k].p && res.pool[k].off == off && res.pool[k].n == cnt) return (int)k;
    return -1;
  };
  auto add_entry = [&](dstack_partition p, int off, int cnt, int* k) -> dstack_status {
    void* sp = nullptr;
    dstack_status s = dstack_partition_query(p, nullptr, nullptr, &sp);
    if (s != DSTACK_OK) {
      dstack_partition_destroy(p);
      return s;
    }
    *k = -1;
    for (size_t q = 0; q < res.pool.size() && *k < 0; ++q)
      if (!res.pool[q].p) *k = (int)q;
    if (*k < 0) {
      *k = (int)res.pool.size();
      res.pool.emplace_back();
    }
    res.pool[*k] = PoolEntry{off, cnt, 0, p, (hipStream_t)sp};
    return DSTACK_OK;
  };
  auto attach = [&](int i, int k) {
    cur[i] = k;
    res.pool[k].users += 1;
    part[i] = res.pool[k].p;
    stream[i] = res.pool[k].s;
  };
  auto detach = [&](int i) {  // model i's last job on its entry has completed
    PoolEntry& e = res.pool[cur[i]];
    if (--e.users == 0) {
      if (res.worker)
        res.worker->destroy(e.p);
      else
        dstack_partition_destroy(e.p);
      e = PoolEntry{};
    }
    cur[i] = -1;
    part[i] = nullptr;
    stream[i] = nullptr;
  };
  for (int i = 0; i < n; ++i) {
    const int off = temporal ? 0 : plan->home_offset[i], cnt = temporal ? prm->total_slots : plan->deployed_slots[i];
    int k = find_entry(off, cnt);
    if (k < 0) {
      dstack_partition p = nullptr;
      st = dstack_partition_create_at(off, cnt, &p);
      if (st != DSTACK_OK) return st;
      st = add_entry(p, off, cnt, &k);
      if (st != DSTACK_OK) return st;
    }
    attach(i, k);
    DS_HIP(hipEventCreate(&res.ev0[i]));
    DS_HIP(hipEventCreate(&res.ev1[i]));
  }
  LaunchState ls(tables, n, prm, sim, plan);

  // warm-up: every batch a job of this run can take (captures its graph);
  // with GPU% changes on, also the graphs of the next kResizeAhead larger
  // GPU% each model can move to (captured only), so that a change needs a
  // new stream and nothing else
  for (int i = 0; i < n; ++i) {
    const int slots = temporal ? prm->total_slots : plan->deployed_slots[i];
    for (int b : kGrid) {
      if (b > tables[i].max_batch) continue;
      if ((temporal || b != plan->batch[i]) && ls.table_latency(i, b, slots) <= 0) continue;
      for (int r = 0; r < 2; ++r) {
        st = launcher_infer(models[i], b, d_in[i], d_out[i], part[i], kLauncherWsBase + i);
        if (st != DSTACK_OK) return st;
      }
    }
    if (temporal || sim->resize_violations <= 0) continue;
    int cur = slots;
    for (int step = 0; step < kResizeAhead; ++step) {
      int next = -1;  // the rule of LaunchState::note_late
      for (int q = 0; q < tables[i].n_slots && next < 0; ++q)
        if (tables[i].slots[q] > cur && tables[i].slots[q] <= prm->total_slots &&
            ls.table_latency(i, plan->batch[i], tables[i].slots[q]) > 0)
          next = tables[i].slots[q];
      if (next < 0) break;
      for (int b : kGrid) {
        if (b > tables[i].max_batch || (b != plan->batch[i] && ls.table_latency(i, b, next) <= 0)) continue;
        st = launcher_prepare(models[i], b, d_in[i], d_out[i], part[i], next * DSTACK_CUS_PER_SLOT,
                              kLauncherWsBase + i);
        if (st != DSTACK_OK) return st;
      }
      cur = next;
    }
  }
  for (const PoolEntry& e : res.pool) {
    if (!e.p) continue;
    st = dstack_synchronize(e.p);
    if (st != DSTACK_OK) return st;
  }

  // streams of a model's next range, created (and unused ones destroyed) by
  // the helper thread; the partitions live in the process (this launcher's
  // and any other), less those queued for destruction (which run first),
  // plus those queued for creation, stay within the library's limit
  {
    int dev = 0;
    DS_HIP(hipGetDevice(&dev));
    res.worker.reset(new PartitionWorker(dev));
  }
  // Read in this order, a task that finishes between the reads can only make
  // the result smaller: a creation counts as live before it leaves creates(),
  // a destruction leaves destroys() before it stops counting as live.
  auto room = [&]() {
    const int c = res.worker->creates();
    int live = 0, max_live = 0;
    dstack_partition_count(&live, &max_live);
    const int d = res.worker->destroys();
    return max_live - live - c + d;
  };
  auto start_create = [&](int i, int off, int cnt) -> dstack_status {
    res.made_off[i] = off;
    res.made_n[i] = cnt;
    res.pending[i] = res.worker->create(off, cnt);
    return DSTACK_OK;
  };
  auto collect = [&](int i, bool wait) -> dstack_status {  // a finished creation into made[i]
    if (!res.pending[i].valid()) return DSTACK_OK;
    if (!wait && res.pending[i].wait_for(std::chrono::seconds(0)) != std::future_status::ready) return DSTACK_OK;
    const NewPartition np = res.pending[i].get();
    if (np.first != DSTACK_OK) return fail(np.first, np.err);
    res.made[i] = np.second;
    return DSTACK_OK;
  };
  auto drop_standby = [&](int i) -> dstack_status {  // an unused stream of model i's
    dstack_status s = collect(i, true);
    if (s != DSTACK_OK) return s;
    if (res.made[i]) res.worker->destroy(res.made[i]);
    res.made[i] = nullptr;
    res.made_off[i] = -1;
    res.made_n[i] = 0;
    return DSTACK_OK;
  };
  std::vector<char> switching(n, 0);  // model i waits for its new range's stream
  // model i is at risk of its next GPU% change (a request late since its last
  // change, or one that waited more than half its SLO before its job
  // started): the stream of its next range as a standby, if there is room
  auto standby = [&](int i) -> dstack_status {
    if (temporal || sim->resize_violations <= 0 || switching[i] || res.pending[i].valid() || res.made[i] ||
        room() < 1)
      return DSTACK_OK;
    int home = 0, dep = 0;
    if (!ls.next_range(i, &home, &dep) || find_entry(home, dep) >= 0) return DSTACK_OK;
    return start_create(i, home, dep);
  };

  const int64_t D = sim->duration_us;
  const int total = prm->total_slots;
  std::vector<Running> run(n);
  std::vector<int64_t> served(n, 0), late(n, 0), pruns(n, 0), fruns(n, 0), skips(n, 0), busy(n, 0);
  std::vector<std::vector<int64_t>> lats(n);
  std::vector<int> next_arr(n, 0);
  size_t next_plan = 0;
  int64_t slot_us = 0, last_end = 0;
  uint64_t h = 0xcbf29ce484222325ULL;
  int jobs = 0, n_ev = 0;
  // planned starts of the session plan (D-STACK) or slice starts (temporal)
  const std::vector<PlannedStart>& P = temporal ? ls.slice_starts() : ls.planned();
  const int64_t t0 = host_us();
  auto clock = [&] { return host_us() - t0; };
  auto note = [&](int64_t t, int kind, int model, int64_t value, uint64_t mask) {
    if (n_ev < event_capacity) events[n_ev] = dstack_serve_event{t, value, mask, kind, model};
    ++n_ev;
  };

  auto launch = [&](int64_t t, int i, uint64_t mask, int64_t table_us, int b, int kind) -> dstack_status {
    Running& r = run[i];
    r.reqs = ls.start(t, i, mask, table_us, b);
    if (!r.reqs.empty() && t - r.reqs.front() > tables[i].slo_us / 2) {  // (requests leave in arrival order)
      dstack_status s = standby(i);
      if (s != DSTACK_OK) return s;
    }
    r.on = true;
    r.start = t;
    r.table_us = table_us;
    r.mask = mask;
    r.batch = b;
    r.kind = kind;
    DS_HIP(hipEventRecord(res.ev0[i], stream[i]));
    dstack_status s = launcher_infer(models[i], b, d_in[i], d_out[i], part[i], kLauncherWsBase + i);
    if (s != DSTACK_OK) return s;
    DS_HIP(hipEventRecord(res.ev1[i], stream[i]));
    for (int64_t v : {t, (int64_t)i, (int64_t)b, (int64_t)mask, table_us, (int64_t)kind})
      for (int k = 0; k < 8; ++k) {
        h ^= ((uint64_t)v >> (8 * k)) & 0xff;
        h *= 0x100000001b3ULL;
      }
    (kind == 0 ? pruns : fruns)[i] += 1;
    return DSTACK_OK;
  };
  auto fod_pass = [&](int64_t t) -> dstack_status {
    LaunchState::Pick pk;
    if (temporal) {
      if (ls.temporal_pick(t, &pk)) return launch(t, pk.model, pk.mask, pk.latency, pk.batch, 0);
    } else if (sim->fod && ls.fod_pick(t, &pk)) {
      return launch(t, pk.model, pk.mask, pk.latency, pk.batch, 1);
    }
    return DSTACK_OK;
  };

  // every decision and launch reads the clock when it is taken, so that a
  // job's start is never before the completion that freed its slots
  for (;;) {
    const int64_t t = clock();
    bool busy_now = false;
    // completions
    for (int i = 0; i < n; ++i) {
      if (!run[i].on) continue;
      const hipError_t q = hipEventQuery(res.ev1[i]);
      if (q == hipErrorNotReady) {
        busy_now = true;
        continue;
      }
      if (q != hipSuccess) {
        res.drained = false;
        return fail(DSTACK_E_HIP, std::string("serve: ") + hipGetErrorString(q));
      }
      float ms = 0.f;
      DS_HIP(hipEventElapsedTime(&ms, res.ev0[i], res.ev1[i]));
      const int64_t gpu_us = (int64_t)llround((double)ms * 1000.0);
      const int64_t te = clock();
      Running& r = run[i];
      r.on = false;
      ls.finish(i);
      int64_t job_late = 0;
      for (int64_t a : r.reqs) {
        served[i] += 1;
        lats[i].push_back(te - a);
        if (te - a > tables[i].slo_us) job_late += 1;
      }
      const int64_t late_since = ls.late_at_end(i, r.start, te, r.reqs);
      late[i] += job_late;
      busy[i] += gpu_us;
      slot_us += (int64_t)__builtin_popcountll(r.mask) * std::max<int64_t>(0, std::min(r.start + gpu_us, D) - r.start);
      last_end = std::max(last_end, te);
      if (jobs < log_capacity)
        log[jobs] = dstack_job_record{r.start, te, gpu_us, r.table_us, i, r.batch, r.kind, r.mask};
      ++jobs;
      note(te, 0, i, 0, 0);
      if (ls.note_late(te, i, late_since)) {
        // GPU% change between batches: the model's next jobs run over its
        // larger range, on the stream of that range if one exists (another
        // model's, or its standby), else on a new one created on a helper
        // thread while the other models keep running (the old stream goes
        // first if nothing else uses it, and an unused standby of another
        // model if the limit needs the room).  Weights, workspace and the
        // graphs captured for that size at warm-up belong to the model and
        // carry over.
        ls.unavailable(i);
        switching[i] = 1;
        const int home = ls.home(i), dep = ls.deployed(i);
        const bool have = find_entry(home, dep) >= 0 ||
                          (res.made_off[i] == home && res.made_n[i] == dep && (res.pending[i].valid() || res.made[i]));
        if (!have) {
          st = drop_standby(i);
          if (st != DSTACK_OK) return st;
          detach(i);
          for (int j = 0; j < n && room() < 1; ++j)
            if (j != i && !switching[j]) {
              st = drop_standby(j);
              if (st != DSTACK_OK) return st;
            }
          st = start_create(i, home, dep);
          if (st != DSTACK_OK) return st;
        }
      } else if (ls.late_count(i) > 0) {
        st = standby(i);
        if (st != DSTACK_OK) return st;
      }
      st = fod_pass(te);
      if (st != DSTACK_OK) return st;
    }
    // GPU% changes whose stream is ready
    for (int i = 0; i < n; ++i) {
      st = collect(i, false);
      if (st != DSTACK_OK) return st;
      if (!switching[i]) continue;
      const int home = ls.home(i), dep = ls.deployed(i);
      int k = find_entry(home, dep);
      if (k < 0) {
        if (!res.made[i]) continue;  // still being created
        st = add_entry(res.made[i], home, dep, &k);
        res.made[i] = nullptr;
        res.made_off[i] = -1;
        if (st != DSTACK_OK) return st;
      } else {
        st = drop_standby(i);  // (a stream of that range came about meanwhile)
        if (st != DSTACK_OK) return st;
      }
      if (cur[i] >= 0) detach(i);
      attach(i, k);
      switching[i] = 0;
      const int64_t tn = clock();
      ls.ready(i, tn);
      note(tn, 3, i, 0, range_mask(home, dep));
      st = fod_pass(tn);
      if (st != DSTACK_OK) return st;
    }
    // planned starts (temporal: slice starts) that are due
    while (next_plan < P.size() && P[next_plan].t <= t) {
      const PlannedStart ps = ls.current(P[next_plan++]);
      const int i = ps.model;
      const int64_t tn = clock();
      note(tn, 1, i, ps.t, ps.mask);
      if (temporal) {
        st = fod_pass(tn);
        if (st != DSTACK_OK) return st;
      } else if (ls.queued(i) && !ls.running(i) && ls.available(i) && ls.free(ps.mask)) {
        st = launch(tn, i, ps.mask, ps.dur, std::min<int>(ls.plan_batch(i), (int)ls.queued(i)), 0);
        if (st != DSTACK_OK) return st;
        busy_now = true;
      } else {
        skips[i] += 1;
      }
    }
    // arrivals that are due, in time order
    for (;;) {
      int j = -1;
      for (int i = 0; i < n; ++i)
        if (next_arr[i] < sim->n_arrivals[i] && sim->arrivals_us[i][next_arr[i]] <= t &&
            (j < 0 || sim->arrivals_us[i][next_arr[i]] < sim->arrivals_us[j][next_arr[j]]))
          j = i;
      if (j < 0) break;
      const int64_t a = sim->arrivals_us[j][next_arr[j]];
      ls.arrive(j, a);
      next_arr[j] += 1;
      const int64_t tn = clock();
      note(tn, 2, j, a, 0);
      st = fod_pass(tn);
      if (st != DSTACK_OK) return st;
    }
    for (int i = 0; i < n; ++i) busy_now = busy_now || run[i].on || switching[i];
    if (t >= D && !busy_now) break;
    if (t > D + kDrainLimitUs) {
      res.drained = false;
      return fail(DSTACK_E_HIP, "serve: a job did not complete within 60 s after the trace");
    }
  }
  for (const PoolEntry& e : res.pool) {
    if (!e.p) continue;
    st = dstack_synchronize(e.p);
    if (st != DSTACK_OK) return st;
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
    s.final_slots = temporal ? total : ls.deployed(i);
  }
  out->utilisation_ppm = (int64_t)((unsigned __int128)slot_us * 1000000 / ((unsigned __int128)total * (uint64_t)D));
  out->job_hash = h;
  out->last_end_us = last_end;
  if (n_log) *n_log = jobs;
  if (n_events) *n_events = n_ev;
  return DSTACK_OK;
}

}  // namespace dstack
