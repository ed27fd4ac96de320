// Host-side scheduling decisions (pure integer functions of a timing table).
#pragma once
#include "common.hpp"

namespace dstack {

// eta(b1, L1, s1) > eta(b2, L2, s2) for eta = b / (L^2 * s), exact.
bool eta_greater(int64_t b1, int64_t L1, int64_t s1, int64_t b2, int64_t L2, int64_t s2);
// argmax over entries with lat > 0 of eta; ties to fewer slots; -1 if none.
int knee_index(int b, const int64_t* lat, const int* slots, int n);
// home placement: offset of each model's fixed range (sizes in slots)
void home_offsets(const int* sizes, int n, int total, int* offs);
uint64_t range_mask(int offset, int size);
dstack_status schedule(const dstack_sched_model* models, int n, const dstack_sched_params* prm,
                       dstack_schedule_out* out);
dstack_status simulate(const dstack_sched_model* models, int n, const dstack_sched_params* prm,
                       const dstack_sim_params* sim, dstack_run_out* out);

}  // namespace dstack
