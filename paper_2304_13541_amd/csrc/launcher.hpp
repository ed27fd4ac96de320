// Decision state of the launcher, shared by the virtual-clock simulation
// and the live launcher: per-model request queues, the slots in use, the
// per-session run counts and busy time that rank the fair, opportunistic,
// dynamic (FOD) fill of Sec. 6.1.2, and the planned starts of the session
// plan repeated every period.  All times are integer microseconds from the
// start of the run; busy time is charged at start with the timing-table
// latency, so that the decisions depend on the table and the arrivals only.
#pragma once
#include <deque>
#include <map>
#include <vector>

#include "sched.hpp"

namespace dstack {

struct PlannedStart {
  int64_t t;
  int model;
  uint64_t mask;
  int64_t dur;
};

class LaunchState {
 public:
  // plan: the dstack_schedule result for the same models and params
  LaunchState(const dstack_sched_model* models, int n, const dstack_sched_params* prm, const dstack_sim_params* sim,
              const dstack_schedule_out* plan);

  const std::vector<PlannedStart>& planned() const { return pstarts_; }
  int n() const { return n_; }
  bool running(int i) const { return running_[i] != 0; }
  bool free(uint64_t mask) const { return (used_ & mask) == 0; }
  size_t queued(int i) const { return queue_[i].size(); }
  void arrive(int i, int64_t t) { queue_[i].push_back(t); }
  int plan_batch(int i) const { return plan_->batch[i]; }

  struct Pick {
    int model;
    uint64_t mask;
    int batch;
    int64_t latency;
  };
  // the FOD choice at time t (false: nothing fits)
  bool fod_pick(int64_t t, Pick* out) const;
  // GPU% change on SLO violations (resize_violations > 0, D-STACK with home
  // placement).  Among the requests of model i that arrived at or after
  // changed_at(i) (earlier ones waited through the previous size and say
  // nothing about the current one), a request counts towards the next change
  // once: when its job starts, if it has waited more than half its SLO by
  // then (the share Eq. meet_half_slo leaves to waiting is used up; start()
  // counts these), else when it completes past its SLO (late_at_end counts
  // these for a job that started at `start` and ended at `end`).  A job of
  // model i ended at t adding `late` such requests: once the count since its
  // last change reaches the threshold the model moves to the next larger
  // swept slot count (true returned) and changed_at(i) becomes t.  Its
  // current size, home offset and the planned job as it now runs:
  bool note_late(int64_t t, int i, int64_t late);
  int64_t late_at_end(int i, int64_t start, int64_t end, const std::vector<int64_t>& reqs) const;
  int64_t changed_at(int i) const { return changed_at_[i]; }
  // the home offset and size model i moves to at its next GPU% change
  // (false: it is at its largest swept share), and the late requests
  // counted towards that change so far
  bool next_range(int i, int* home, int* dep) const;
  int64_t late_count(int i) const { return viol_[i]; }
  // the live launcher: model i's new stream is being created (it neither
  // starts planned jobs nor is picked by FOD) until ready(i, t), which also
  // moves changed_at(i) to t
  void unavailable(int i) { avail_[i] = 0; }
  void ready(int i, int64_t t) {
    avail_[i] = 1;
    changed_at_[i] = t;
  }
  bool available(int i) const { return avail_[i] != 0; }
  int deployed(int i) const { return dep_[i]; }
  int home(int i) const { return home_[i]; }
  int64_t resizes(int i) const { return resizes_[i]; }
  PlannedStart current(const PlannedStart& ps) const;
  // temporal policy: the slice starts in time order, and the job its slice
  // owner starts at time t on the whole GPU (false: none)
  const std::vector<PlannedStart>& slice_starts() const { return slices_; }
  bool temporal_pick(int64_t t, Pick* out) const;
  bool temporal() const { return sim_->policy == 3; }
  bool any_running() const { return used_ != 0; }
  // a job starts: pops b requests (returned, oldest first), charges the run
  // and `charged_us` of busy time, marks its slots used
  std::vector<int64_t> start(int64_t t, int i, uint64_t mask, int64_t charged_us, int b);
  // the job of model i ended: frees its slots
  void finish(int i);
  // latency of batch b at `slots` from the table (largest swept count <= slots), -1 if none
  int64_t table_latency(int i, int b, int slots) const;

 private:
  const dstack_sched_model* models_;
  int n_;
  const dstack_sched_params* prm_;
  const dstack_sim_params* sim_;
  const dstack_schedule_out* plan_;
  int64_t T_, D_;
  std::vector<PlannedStart> pstarts_;  // by time, then plan order
  int64_t cycle_ = 0;                  // temporal policy: slice cycle, slice offsets and lengths
  std::vector<int64_t> slice_off_, slice_len_;
  std::vector<PlannedStart> slices_;
  std::vector<std::deque<int64_t>> queue_;
  std::vector<char> running_;
  std::vector<uint64_t> run_mask_;
  uint64_t used_ = 0;
  std::vector<std::map<int64_t, int64_t>> runs_;  // session -> runs started
  std::vector<int64_t> busy_;
  std::vector<int> dep_, home_;                 // current deployed slots and home offset
  std::vector<int64_t> viol_, resizes_;         // late requests since the last change, changes
  std::vector<int64_t> changed_at_;             // time of the last change (0: none)
  std::vector<char> avail_;                     // 0 while the live launcher builds its new stream
};

// nearest-rank percentile (sorts v)
int64_t nearest_rank(std::vector<int64_t>& v, int pct);
// duration > 0, window >= 1, each model's arrivals sorted inside [0, duration)
bool check_trace(int n, const dstack_sim_params* sim);

dstack_status simulate_ideal(const dstack_ideal_model* models, int n, int64_t horizon, int64_t slot, int total,
                             dstack_ideal_out* out);

// The live launcher's model workspaces: model i of a run uses workspace id
// kLauncherWsBase + i, whose activations, split-K buffers and captured graphs
// belong to the model rather than to a partition, so a GPU% change (a new
// partition) reuses them and allocates, frees and synchronises nothing.
constexpr int kLauncherWsBase = 4, kLauncherWsCount = 4;
// dstack_infer with the launcher workspace ws_id
dstack_status launcher_infer(dstack_model h, int batch, const void* d_in, void* d_out, dstack_partition p, int ws_id);
// records and instantiates the graph of a forward planned for n_cu CUs
// (captured on p's stream, nothing runs), for a later launcher_infer on a
// partition of that size
dstack_status launcher_prepare(dstack_model h, int batch, const void* d_in, void* d_out, dstack_partition p, int n_cu,
                               int ws_id);

dstack_status serve(const dstack_model* models, int n, const void* const* d_in, void* const* d_out,
                    const dstack_sched_model* tables, const dstack_sched_params* prm, const dstack_sim_params* sim,
                    dstack_run_out* out, dstack_job_record* log, int log_capacity, int* n_log,
                    dstack_serve_event* events, int event_capacity, int* n_events);

}  // namespace dstack
