// Host-side scheduling decisions (pure integer functions of a timing table).
#pragma once
#include <functional>
#include <utility>
#include <vector>

#include "common.hpp"

namespace dstack {

// eta(b1, L1, s1) > eta(b2, L2, s2) for eta = b / (L^2 * s), exact.
bool eta_greater(int64_t b1, int64_t L1, int64_t s1, int64_t b2, int64_t L2, int64_t s2);
// argmax over entries with lat > 0 of eta; ties to fewer slots; -1 if none.
int knee_index(int b, const int64_t* lat, const int* slots, int n);
// Knee search for a model without a profile (Sec. 3.6): over the ascending
// candidate slot counts cand, starting at the last candidate <= start,
// compare eta(cand[i]) with eta(cand[i + 1]) and keep the half where eta
// rises (ties: fewer slots) until one candidate is left; returns its index.
// latency(s) > 0 is the measured latency at s slots, called once per
// distinct s; probes receives (s, latency) in call order.
int knee_search(int b, const std::vector<int>& cand, int start, const std::function<int64_t(int)>& latency,
                std::vector<std::pair<int, int64_t>>* probes);
// home placement: offset of each model's fixed range (sizes in slots)
void home_offsets(const int* sizes, int n, int total, int* offs);
uint64_t range_mask(int offset, int size);
dstack_status schedule(const dstack_sched_model* models, int n, const dstack_sched_params* prm,
                       dstack_schedule_out* out);
dstack_status simulate(const dstack_sched_model* models, int n, const dstack_sched_params* prm,
                       const dstack_sim_params* sim, dstack_run_out* out);

}  // namespace dstack
