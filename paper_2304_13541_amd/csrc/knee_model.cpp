// Analytical DNN latency model and its knee (Sec. 4.3), host only.
//
// A DNN is a sequence of kernels; kernel i has N_i parallelizable operations
// of t_p each (Eq. layer_num_ops generates the paper's synthetic sequence),
// runs in E_i = N_i t_p / max(1, min(S, N_i)) on S SMs (CUs here; Eq.
// execution_time_per_layer), repeats R_i times and waits t_np plus E_m for
// its start and its data (Eqs. memory_latency, total_non_paralleizable_time).
// E_t = W_se + sum_i R_i E_i (Eq. total_time_shrinking_kernel); the most
// efficient S maximises 1 / (E_t^2 S) (Eq. first_order_derivative).
//
// Readings: N_i is clamped at 0 once the decrement reaches it; E_m is
// d_i / (M S) with M the bandwidth per SM (the total grows with S, as the
// text states); t_p may differ per kernel.  The sums run in kernel order and
// this file is built without floating-point contraction, so results are
// reproducible to the bit.
#include <algorithm>
#include <cmath>

#include "common.hpp"

namespace dstack {

static double km_kernel_time(double n, double tp, int s) { return n * tp / std::max(1.0, std::min((double)s, n)); }

static double km_memory_time(double d, double m, int s) { return m <= 0.0 ? 0.0 : d / (m * (double)s); }

static double km_total_time(const dstack_knee_model& km, int s) {
  double w_se = 0.0;
  for (int i = 0; i < km.n_kernels; ++i) {
    const double r = km.reps ? km.reps[i] : 1.0;
    const double em = km.data ? km_memory_time(km.data[i], km.mem_bw_per_sm, s) : 0.0;
    w_se += r * (km.t_np + em);
  }
  w_se *= km.batch_serial;
  double par = 0.0;
  for (int i = 0; i < km.n_kernels; ++i) {
    const double r = km.reps ? km.reps[i] : 1.0;
    par += r * km_kernel_time(km.n_par[i], km.t_p[i], s);
  }
  return w_se + par;
}

dstack_status knee_model_sequence(int p, int b, int kmax, double* n_out) {
  DS_CHECK(n_out, DSTACK_E_INVALID, "knee_model_sequence: null output");
  DS_CHECK(p >= 0 && b >= 1 && kmax >= 1 && (long)p * b < (1L << 40), DSTACK_E_INVALID,
           "knee_model_sequence: p >= 0, b >= 1, kmax >= 1");
  const double pb = (double)((long)p * b);
  const double step = pb / (double)kmax;
  n_out[0] = pb;
  for (int i = 1; i < kmax; ++i) n_out[i] = std::max(0.0, std::floor(n_out[i - 1] - step));
  return DSTACK_OK;
}

dstack_status knee_model_eval(const dstack_knee_model* km, const int* s_values, int n_s, double* et_out,
                              int* knee_index) {
  DS_CHECK(km && s_values && et_out && knee_index && km->n_par && km->t_p, DSTACK_E_INVALID,
           "knee_model_eval: null pointer");
  DS_CHECK(km->n_kernels >= 1 && n_s >= 1, DSTACK_E_INVALID, "knee_model_eval: no kernels or no candidates");
  for (int i = 0; i < km->n_kernels; ++i) {
    DS_CHECK(std::isfinite(km->n_par[i]) && km->n_par[i] >= 0.0 && std::isfinite(km->t_p[i]) && km->t_p[i] >= 0.0,
             DSTACK_E_INVALID, "knee_model_eval: N_i and t_p must be finite and >= 0");
    DS_CHECK(!km->reps || (std::isfinite(km->reps[i]) && km->reps[i] >= 0.0), DSTACK_E_INVALID,
             "knee_model_eval: R_i must be finite and >= 0");
    DS_CHECK(!km->data || (std::isfinite(km->data[i]) && km->data[i] >= 0.0), DSTACK_E_INVALID,
             "knee_model_eval: d_i must be finite and >= 0");
  }
  DS_CHECK(std::isfinite(km->t_np) && km->t_np >= 0.0 && std::isfinite(km->batch_serial) &&
               km->batch_serial >= 0.0 && std::isfinite(km->mem_bw_per_sm),
           DSTACK_E_INVALID, "knee_model_eval: t_np, b and M must be finite (t_np, b >= 0)");
  for (int j = 0; j < n_s; ++j) DS_CHECK(s_values[j] >= 1, DSTACK_E_INVALID, "knee_model_eval: S must be >= 1");
  double best = 0.0;
  int arg = -1;
  for (int j = 0; j < n_s; ++j) {
    const double et = km_total_time(*km, s_values[j]);
    et_out[j] = et;
    const double v = et * et * (double)s_values[j];
    if (arg < 0 || v < best) {
      best = v;
      arg = j;
    }
  }
  *knee_index = arg;
  return DSTACK_OK;
}

}  // namespace dstack
